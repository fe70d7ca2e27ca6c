// Host-side check of the library under AddressSanitizer and UndefinedBehaviorSanitizer.
//
// Reads model descriptors dumped by the test (the raw bytes of mopar_tensor_desc /
// mopar_op arrays, see test_host_sanitizers.py) and drives every host-only entry point:
// model creation and validation (valid and corrupted descriptors), the layer profiles,
// planning over them, workspace sizing, cut tensors, codec sizes, timing slots; then the
// planner and sub-slice ranges on random inputs.  No device call is made.  Exit status 0
// when every call returned what was expected.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

#include "../../include/mopar.h"

static int failures = 0;
#define CHECK(cond)                                                                  \
    do {                                                                             \
        if (!(cond)) {                                                               \
            std::fprintf(stderr, "check failed: %s (line %d)\n", #cond, __LINE__);   \
            ++failures;                                                              \
        }                                                                            \
    } while (0)

struct Dump {
    int32_t expect_ok, dtype, n_tensors, n_ops, n_layers, input, output;
    int64_t weights_bytes;
    std::vector<mopar_tensor_desc> tensors;
    std::vector<mopar_op> ops;
};

static bool read_dump(const char* path, Dump& d) {
    FILE* f = std::fopen(path, "rb");
    if (!f) return false;
    char magic[4];
    int32_t hdr[8];
    bool ok = std::fread(magic, 1, 4, f) == 4 && std::memcmp(magic, "MOPD", 4) == 0 &&
              std::fread(hdr, sizeof(int32_t), 8, f) == 8 && hdr[0] == 1 &&
              hdr[7] == static_cast<int32_t>(sizeof(mopar_tensor_desc) * 1000 + sizeof(mopar_op));
    if (ok) {
        d.expect_ok = hdr[1], d.dtype = hdr[2], d.n_tensors = hdr[3], d.n_ops = hdr[4], d.n_layers = hdr[5],
        d.input = hdr[6];
        ok = std::fread(&d.output, sizeof(int32_t), 1, f) == 1 && std::fread(&d.weights_bytes, 8, 1, f) == 1 &&
             d.n_tensors >= 0 && d.n_ops >= 0 && d.n_tensors < 100000 && d.n_ops < 100000;
    }
    if (ok) {
        d.tensors.resize(d.n_tensors);
        d.ops.resize(d.n_ops);
        ok = std::fread(d.tensors.data(), sizeof(mopar_tensor_desc), d.n_tensors, f) ==
                 static_cast<size_t>(d.n_tensors) &&
             std::fread(d.ops.data(), sizeof(mopar_op), d.n_ops, f) == static_cast<size_t>(d.n_ops);
    }
    std::fclose(f);
    return ok;
}

static void drive_model(const Dump& d, const char* path) {
    mopar_model_desc desc{};
    desc.dtype = d.dtype;
    desc.n_tensors = d.n_tensors;
    desc.tensors = d.tensors.data();
    desc.n_ops = d.n_ops;
    desc.ops = d.ops.data();
    desc.n_layers = d.n_layers;
    desc.input = d.input;
    desc.output = d.output;
    // the weights are never dereferenced on the host: any non-null address does
    static unsigned char dummy[16];
    mopar_model_t m = nullptr;
    const int rc = mopar_model_create(&desc, dummy, static_cast<size_t>(d.weights_bytes), &m);
    if (d.expect_ok == 2 && rc != MOPAR_OK) return;   // fuzzed descriptor: either outcome is fine
    if (!d.expect_ok) {
        CHECK(rc != MOPAR_OK && m == nullptr && std::strlen(mopar_last_error()) > 0);
        if (rc == MOPAR_OK) std::fprintf(stderr, "%s: an invalid model was accepted\n", path);
        mopar_model_destroy(m);
        return;
    }
    CHECK(rc == MOPAR_OK);
    if (rc != MOPAR_OK) {
        std::fprintf(stderr, "%s: %s\n", path, mopar_last_error());
        return;
    }
    const int n = d.n_layers;
    std::vector<mopar_layer_profile> prof(n), dom(n);
    CHECK(mopar_model_profile(m, prof.data()) == MOPAR_OK);
    CHECK(mopar_model_profile_dominant(m, 0.8, dom.data()) == MOPAR_OK);
    CHECK(mopar_model_profile_dominant(m, 0.0, dom.data()) != MOPAR_OK);
    CHECK(mopar_model_profile_dominant(m, 1.5, dom.data()) != MOPAR_OK);
    for (int l = 0; l < n; ++l) CHECK(prof[l].mem_bytes > 0 && prof[l].time_s > 0 && prof[l].out_bytes > 0);
    // plans in free mode and with every slice count, then everything a plan sizes
    for (int ns = 0; ns <= n; ++ns) {
        std::vector<int32_t> ends(n), ks(n);
        mopar_plan_opts o{};
        o.n_slices = ns;
        o.k_max = 4;
        o.elim_tau = ns == 0 ? 0.05 : -1.0;
        o.c_m = 1.0;
        o.c_n = 1.0;
        o.bw_Bps = 8e12;
        mopar_plan p{};
        p.n_layers = n;
        p.slice_end = ends.data();
        p.k = ks.data();
        const int prc = mopar_plan_slices(prof.data(), n, &o, &p);
        if (prc != MOPAR_OK) {
            CHECK(prc == MOPAR_E_INFEASIBLE);
            continue;
        }
        size_t ws = 0;
        CHECK(mopar_model_workspace_bytes(m, &p, &ws) == MOPAR_OK);
        size_t pws = 0;
        CHECK(mopar_pipeline_workspace_bytes(m, &p, 3, &pws) == MOPAR_OK);
        CHECK(pws >= 3 * ws);
        for (int s = 0; s + 1 < p.n_slices; ++s) {
            int32_t cnt = 0;
            CHECK(mopar_model_cut_tensors(m, p.slice_end[s], nullptr, 0, &cnt) == MOPAR_OK && cnt >= 1);
            std::vector<int32_t> tids(cnt > 0 ? cnt : 1);
            CHECK(mopar_model_cut_tensors(m, p.slice_end[s], tids.data(), cnt, &cnt) == MOPAR_OK);
            for (int q = 0; q < cnt; ++q) {
                const mopar_tensor_desc& t = d.tensors[tids[q]];
                mopar_codec raw{};
                raw.kind = MOPAR_CODEC_RAW;
                size_t bytes = 0;
                CHECK(mopar_boundary_code_bytes(&raw, &t, &bytes) == MOPAR_OK && bytes > 0);
                mopar_codec ae{};
                ae.kind = MOPAR_CODEC_AE;
                ae.c = static_cast<int32_t>(t.rank == 4 ? t.dims[1] : t.dims[t.rank - 1]);
                ae.c_code = ae.c >= 8 ? ae.c / 8 : 1;
                ae.w_enc = ae.w_dec = dummy;
                CHECK(mopar_boundary_code_bytes(&ae, &t, &bytes) == MOPAR_OK);
                ae.c += 1;   // channels that do not match the tensor's
                CHECK(mopar_boundary_code_bytes(&ae, &t, &bytes) == MOPAR_E_SHAPE);
            }
        }
        // a plan for another node count and an invalid k are refused
        p.n_layers = n + 1;
        CHECK(mopar_model_workspace_bytes(m, &p, &ws) != MOPAR_OK);
        p.n_layers = n;
        ks[0] = 1 << 30;
        CHECK(mopar_model_workspace_bytes(m, &p, &ws) != MOPAR_OK);
    }
    int32_t cnt = 0;
    CHECK(mopar_model_cut_tensors(m, n - 1, nullptr, 0, &cnt) != MOPAR_OK);
    CHECK(mopar_model_cut_tensors(m, -1, nullptr, 0, &cnt) != MOPAR_OK);
    int32_t slots = 0;
    CHECK(mopar_model_timing_slots(m, &slots) == MOPAR_OK && slots == d.n_ops + 2 * (n - 1));
    CHECK(mopar_model_set_timing(m, 1) == MOPAR_OK);
    CHECK(mopar_model_set_timing(m, 0) == MOPAR_OK);
    mopar_model_destroy(m);
}

static void drive_planner(unsigned seed) {
    std::mt19937 rng(seed);
    std::uniform_real_distribution<double> u(0.0, 1.0);
    for (int trial = 0; trial < 3000; ++trial) {
        const int n = 1 + static_cast<int>(rng() % 40);
        std::vector<mopar_layer_profile> prof(n);
        for (auto& l : prof) {
            l.mem_bytes = 1 + 1e6 * u(rng);
            l.time_s = 1e-6 + 1e-3 * u(rng);
            l.out_bytes = 1 + 1e6 * u(rng);
            l.rd_width = (rng() % 3) ? static_cast<int32_t>(rng() % 64) : 0;
        }
        const int kmax = 1 + static_cast<int>(rng() % 8);
        std::vector<uint8_t> allowed(n > 1 ? n - 1 : 1);
        for (auto& a : allowed) a = static_cast<uint8_t>(rng() % 2);
        std::vector<double> ratio(n > 1 ? n - 1 : 1), tp(n * kmax), ta(n * kmax);
        for (auto& r : ratio) r = 1.0 + 63.0 * u(rng);
        for (auto& v : tp) v = 1e-3 * u(rng);
        for (auto& v : ta) v = 1e-4 * u(rng);
        std::vector<int32_t> kov(n);
        for (auto& k : kov) k = (rng() % 5 == 0) ? static_cast<int32_t>(rng() % 5) : 0;
        mopar_plan_opts o{};
        o.n_slices = static_cast<int32_t>(rng() % (n + 2)) - (rng() % 10 == 0 ? 1 : 0);
        o.k_max = kmax;
        o.allowed_cut = (rng() % 2) ? allowed.data() : nullptr;
        o.elim_tau = (rng() % 2) ? 0.05 : -1.0;
        o.c_m = u(rng);
        o.c_n = u(rng);
        o.bw_Bps = (rng() % 20 == 0) ? 0.0 : 1e9 + 1e12 * u(rng);
        o.ratio = (rng() % 2) ? ratio.data() : nullptr;
        o.lambda_bytes = (rng() % 2) ? 1e5 * u(rng) : 0.0;
        o.tp_table = (rng() % 2) ? tp.data() : nullptr;
        o.ta_table = o.tp_table && (rng() % 2) ? ta.data() : nullptr;
        o.k_override = (rng() % 3 == 0) ? kov.data() : nullptr;
        o.uniform = (rng() % 6 == 0) ? 1 : 0;
        std::vector<int32_t> ends(n), ks(n);
        mopar_plan p{};
        p.n_layers = (rng() % 30 == 0) ? n - 1 : n;
        p.slice_end = ends.data();
        p.k = ks.data();
        const int rc = mopar_plan_slices(prof.data(), n, &o, &p);
        if (rc == MOPAR_OK) {
            CHECK(p.n_slices >= 1 && p.n_slices <= n && p.slice_end[p.n_slices - 1] == n - 1);
            for (int s = 1; s < p.n_slices; ++s) CHECK(p.slice_end[s] > p.slice_end[s - 1]);
            for (int l = 0; l < n; ++l) CHECK(p.k[l] >= 1);
        } else {
            CHECK(std::strlen(mopar_last_error()) > 0);
        }
    }
    CHECK(mopar_plan_slices(nullptr, 3, nullptr, nullptr) == MOPAR_E_ARG);
    {   // a forced k beyond k_max has no measured time: refused, never read past the tables
        std::vector<mopar_layer_profile> prof(3, mopar_layer_profile{1e6, 1e-4, 1e3, 64, 0});
        std::vector<double> tp(3 * 2, 1e-4);
        std::vector<int32_t> kov{0, 4, 0}, ends(3), ks(3);
        mopar_plan_opts o{};
        o.k_max = 2;
        o.bw_Bps = 1e12;
        o.tp_table = tp.data();
        o.k_override = kov.data();
        mopar_plan p{};
        p.n_layers = 3;
        p.slice_end = ends.data();
        p.k = ks.data();
        CHECK(mopar_plan_slices(prof.data(), 3, &o, &p) == MOPAR_E_ARG);
        o.tp_table = nullptr;
        CHECK(mopar_plan_slices(prof.data(), 3, &o, &p) == MOPAR_OK && p.k[1] == 4);
    }
    for (int nn = -2; nn < 70; ++nn)
        for (int k = -1; k < 10; ++k)
            for (int j = -1; j < 11; ++j) {
                int32_t lo = -7, hi = -7;
                const int rc = mopar_subslice_range(nn, k, j, &lo, &hi);
                if (rc == MOPAR_OK) CHECK(0 <= lo && lo <= hi && hi <= nn);
            }
}

int main(int argc, char** argv) {
    for (int i = 1; i < argc; ++i) {
        Dump d;
        if (!read_dump(argv[i], d)) {
            std::fprintf(stderr, "%s: unreadable descriptor dump\n", argv[i]);
            return 2;
        }
        drive_model(d, argv[i]);
    }
    drive_planner(12345u);
    std::printf("%d models, %d failed checks\n", argc - 1, failures);
    return failures == 0 ? 0 : 1;
}
