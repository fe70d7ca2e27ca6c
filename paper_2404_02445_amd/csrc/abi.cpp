// extern "C" entry points: argument checks live in the *_impl functions, this
// file only turns C++ exceptions into status codes and keeps the error text.
#include <exception>
#include <string>

#include "internal.h"

namespace mopar {

int plan_slices_impl(const mopar_layer_profile*, int32_t, const mopar_plan_opts*, mopar_plan*);
int subslice_range_impl(int32_t, int32_t, int32_t, int32_t*, int32_t*);
int model_create_impl(const mopar_model_desc*, const void*, size_t, mopar_model_t*);
void model_destroy_impl(mopar_model_t);
int model_profile_impl(const mopar_model_s*, mopar_layer_profile*, double);
int workspace_bytes_impl(const mopar_model_s*, const mopar_plan*, size_t*);
int slice_forward_impl(const mopar_model_s*, const mopar_plan*, int32_t, const void*, void*, void*, size_t, void*);
int code_bytes_impl(const mopar_codec*, const mopar_tensor_desc*, size_t*);
int encode_impl(const mopar_codec*, const mopar_tensor_desc*, const void*, void*, void*);
int decode_impl(const mopar_codec*, const mopar_tensor_desc*, const void*, void*, void*);
int model_forward_impl(const mopar_model_s*, const mopar_plan*, const mopar_codec*, const void*, void*, void* const*,
                       void*, size_t, void*);
int model_forward_static_impl(const mopar_model_s*, const mopar_plan*, const mopar_codec*, const void*, void*,
                              void* const*, void*);

int pipeline_ws_bytes_impl(const mopar_model_s*, const mopar_plan*, int32_t, size_t*);
int pipeline_create_impl(const mopar_model_s*, const mopar_plan*, const mopar_codec*, int32_t, int32_t, void* const*,
                         void*, size_t, void* const*, mopar_pipeline_t*);
int pipeline_submit_impl(mopar_pipeline_s*, const void*, void*);
int pipeline_use_graphs_impl(mopar_pipeline_s*, int32_t);
void pipeline_destroy_impl(mopar_pipeline_s*);
int set_timing_impl(mopar_model_s*, int32_t);
int timing_slots_impl(const mopar_model_s*, int32_t*);
int op_times_impl(const mopar_model_s*, float*, int32_t);
int cut_tensors_impl(const mopar_model_s*, int32_t, int32_t*, int32_t, int32_t*);
int measure_impl(mopar_model_s*, int32_t, int32_t, const void*, void*, void*, size_t, void*, double*);

static thread_local std::string g_error;

int set_error(int status, const std::string& msg) {
    g_error = msg;
    return status;
}

int hip_check(hipError_t e, const char* what) {
    if (e == hipSuccess) return MOPAR_OK;
    return set_error(MOPAR_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

template <typename F>
static int guarded(const char* who, F&& f) {
    try {
        g_error.clear();
        return f();
    } catch (const std::exception& e) {
        return set_error(MOPAR_E_ARG, std::string(who) + ": " + e.what());
    } catch (...) {
        return set_error(MOPAR_E_ARG, std::string(who) + ": unknown exception");
    }
}

}  // namespace mopar

using namespace mopar;

extern "C" {

int mopar_subslice_range(int32_t n, int32_t k, int32_t j, int32_t* lo, int32_t* hi) {
    return guarded("mopar_subslice_range", [&] { return subslice_range_impl(n, k, j, lo, hi); });
}

int mopar_plan_slices(const mopar_layer_profile* layers, int32_t n, const mopar_plan_opts* opts, mopar_plan* out) {
    return guarded("mopar_plan_slices", [&] { return plan_slices_impl(layers, n, opts, out); });
}

int mopar_model_create(const mopar_model_desc* desc, const void* weights_dev, size_t weights_bytes,
                       mopar_model_t* out) {
    return guarded("mopar_model_create", [&] { return model_create_impl(desc, weights_dev, weights_bytes, out); });
}

void mopar_model_destroy(mopar_model_t model) { model_destroy_impl(model); }

int mopar_model_profile(mopar_model_t model, mopar_layer_profile* out) {
    return guarded("mopar_model_profile", [&] { return model_profile_impl(model, out, 1.0); });
}

int mopar_model_profile_dominant(mopar_model_t model, double frac, mopar_layer_profile* out) {
    return guarded("mopar_model_profile_dominant", [&] { return model_profile_impl(model, out, frac); });
}

int mopar_model_workspace_bytes(mopar_model_t model, const mopar_plan* plan, size_t* bytes) {
    return guarded("mopar_model_workspace_bytes", [&] { return workspace_bytes_impl(model, plan, bytes); });
}

int mopar_slice_forward(mopar_model_t model, const mopar_plan* plan, int32_t s, const void* in_dev, void* out_dev,
                        void* ws, size_t ws_bytes, void* stream) {
    return guarded("mopar_slice_forward",
                   [&] { return slice_forward_impl(model, plan, s, in_dev, out_dev, ws, ws_bytes, stream); });
}

int mopar_boundary_code_bytes(const mopar_codec* codec, const mopar_tensor_desc* x, size_t* bytes) {
    return guarded("mopar_boundary_code_bytes", [&] { return code_bytes_impl(codec, x, bytes); });
}

int mopar_boundary_encode(const mopar_codec* codec, const mopar_tensor_desc* x, const void* x_dev, void* code_dev,
                          void* stream) {
    return guarded("mopar_boundary_encode", [&] { return encode_impl(codec, x, x_dev, code_dev, stream); });
}

int mopar_boundary_decode(const mopar_codec* codec, const mopar_tensor_desc* y, const void* code_dev, void* y_dev,
                          void* stream) {
    return guarded("mopar_boundary_decode", [&] { return decode_impl(codec, y, code_dev, y_dev, stream); });
}

int mopar_model_forward(mopar_model_t model, const mopar_plan* plan, const mopar_codec* codecs, const void* in_dev,
                        void* out_dev, void* const* code_bufs, void* ws, size_t ws_bytes, void* stream) {
    return guarded("mopar_model_forward", [&] {
        return model_forward_impl(model, plan, codecs, in_dev, out_dev, code_bufs, ws, ws_bytes, stream);
    });
}

int mopar_model_forward_static(mopar_model_t model, const mopar_plan* plan, const mopar_codec* codecs,
                               const void* in_dev, void* out_dev, void* const* code_bufs, void* stream) {
    return guarded("mopar_model_forward_static", [&] {
        return model_forward_static_impl(model, plan, codecs, in_dev, out_dev, code_bufs, stream);
    });
}

int mopar_pipeline_workspace_bytes(mopar_model_t model, const mopar_plan* plan, int32_t replicas, size_t* bytes) {
    return guarded("mopar_pipeline_workspace_bytes",
                   [&] { return pipeline_ws_bytes_impl(model, plan, replicas, bytes); });
}

int mopar_pipeline_create(mopar_model_t model, const mopar_plan* plan, const mopar_codec* codecs, int32_t replicas,
                          int32_t depth, void* const* streams, void* ws, size_t ws_bytes, void* const* code_bufs,
                          mopar_pipeline_t* out) {
    return guarded("mopar_pipeline_create", [&] {
        return pipeline_create_impl(model, plan, codecs, replicas, depth, streams, ws, ws_bytes, code_bufs, out);
    });
}

int mopar_pipeline_submit(mopar_pipeline_t pipe, const void* in_dev, void* out_dev) {
    return guarded("mopar_pipeline_submit", [&] { return pipeline_submit_impl(pipe, in_dev, out_dev); });
}

int mopar_pipeline_use_graphs(mopar_pipeline_t pipe, int32_t enable) {
    return guarded("mopar_pipeline_use_graphs", [&] { return pipeline_use_graphs_impl(pipe, enable); });
}

void mopar_pipeline_destroy(mopar_pipeline_t pipe) { pipeline_destroy_impl(pipe); }

int mopar_model_set_timing(mopar_model_t model, int32_t enable) {
    return guarded("mopar_model_set_timing", [&] { return set_timing_impl(model, enable); });
}

int mopar_model_timing_slots(mopar_model_t model, int32_t* n) {
    return guarded("mopar_model_timing_slots", [&] { return timing_slots_impl(model, n); });
}

int mopar_model_op_times(mopar_model_t model, float* ms, int32_t n) {
    return guarded("mopar_model_op_times", [&] { return op_times_impl(model, ms, n); });
}

int mopar_model_cut_tensors(mopar_model_t model, int32_t node, int32_t* tids, int32_t cap, int32_t* count) {
    return guarded("mopar_model_cut_tensors", [&] { return cut_tensors_impl(model, node, tids, cap, count); });
}

int mopar_model_measure(mopar_model_t model, int32_t k_max, int32_t reps, const void* in_dev, void* out_dev,
                        void* ws, size_t ws_bytes, void* stream, double* tp_out) {
    return guarded("mopar_model_measure",
                   [&] { return measure_impl(model, k_max, reps, in_dev, out_dev, ws, ws_bytes, stream, tp_out); });
}

const char* mopar_last_error(void) { return g_error.c_str(); }

const char* mopar_version(void) { return "mopar-mi355x 0.1 (gfx950)"; }

}  // extern "C"
