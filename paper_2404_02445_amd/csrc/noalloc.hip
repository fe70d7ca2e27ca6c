// Sliced forward pass for callers that cannot allocate device memory (code under
// HIP graph capture, serving loops that forbid allocation): the workspace is a
// file-scope device array the library owns -- each GPU holds its own copy for the
// life of the process -- instead of a buffer the caller passes in.
#include <mutex>

#include "internal.h"

namespace mopar {

int model_forward_impl(const mopar_model_s*, const mopar_plan*, const mopar_codec*, const void*, void*, void* const*,
                       void*, size_t, void*);
int workspace_bytes_impl(const mopar_model_s*, const mopar_plan*, size_t*);
bool model_timing_enabled(const mopar_model_s*);

namespace {

constexpr size_t kScratchBytes = MOPAR_STATIC_WORKSPACE_BYTES;
static_assert(kScratchBytes % 256 == 0, "whole 256-byte workspace slots");

// The workspace.  In host code this name is only a stand-in for the symbol: kernels get the
// device address that hipGetSymbolAddress returns for the current GPU.
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};   // device address of `scratch` on each GPU, resolved on first use

// The address of this GPU's copy of `scratch`: looked up once per device, with that device current.
int scratch_on(int dev, void** out) {
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[dev]) {
        int cur = -1;
        int rc = hip_check(hipGetDevice(&cur), "mopar_model_forward_static: hipGetDevice");
        if (rc) return rc;
        if (cur != dev) {
            rc = hip_check(hipSetDevice(dev), "mopar_model_forward_static: hipSetDevice");
            if (rc) return rc;
        }
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev) (void)hipSetDevice(cur);
        rc = hip_check(e, "mopar_model_forward_static: hipGetSymbolAddress");
        if (rc) return rc;
        if (!p) return set_error(MOPAR_E_HIP, "mopar_model_forward_static: null workspace address");
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return MOPAR_OK;
}

}  // namespace

int model_forward_static_impl(const mopar_model_s* m, const mopar_plan* p, const mopar_codec* codecs, const void* in,
                              void* out, void* const* code_bufs, void* stream) {
    size_t need = 0;
    int rc = workspace_bytes_impl(m, p, &need);          // checks model and plan; host only
    if (rc) return rc;
    if (need > kScratchBytes)
        return set_error(MOPAR_E_WORKSPACE, "mopar_model_forward_static: the plan needs " + std::to_string(need) +
                                                " bytes of workspace, the static workspace holds " +
                                                std::to_string(kScratchBytes) +
                                                " (use mopar_model_forward with a caller buffer)");
    if (model_timing_enabled(m))
        return set_error(MOPAR_E_ARG, "mopar_model_forward_static: per-op timing is on (it creates events); "
                                      "disable it with mopar_model_set_timing");
    int dev = 0;
    rc = stream ? hip_check(hipStreamGetDevice(static_cast<hipStream_t>(stream), &dev), "hipStreamGetDevice")
                : hip_check(hipGetDevice(&dev), "hipGetDevice");
    if (rc) return rc;
    if (dev < 0 || dev >= kMaxDevices) return set_error(MOPAR_E_ARG, "mopar_model_forward_static: device index");
    void* ws = nullptr;
    rc = scratch_on(dev, &ws);
    if (rc) return rc;
    return model_forward_impl(m, p, codecs, in, out, code_bufs, ws, kScratchBytes, stream);
}

}  // namespace mopar
