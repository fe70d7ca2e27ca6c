// Internal declarations shared by the host code and the kernel launchers.
#pragma once

#include <cstdint>
#include <string>
#include <utility>
#include <vector>

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "../../include/mopar.h"

namespace mopar {

// Thread-local error text; set_error returns the status for `return set_error(...)`.
int set_error(int status, const std::string& msg);
int hip_check(hipError_t e, const char* what);

// ---------------------------------------------------------------------------
// Kernel launches.  While a model measures op times, the calling thread has a
// LaunchTimer: every kernel is then launched with its own start / stop event
// pair, stamped by the runtime with that kernel's begin and end, so an op's time
// is the sum of its kernels' durations (launch gaps excluded).
// ---------------------------------------------------------------------------
struct LaunchTimer {
    std::vector<std::pair<hipEvent_t, hipEvent_t>>* pool;   // grows on demand, owned by the model
    size_t* next;                                           // next unused pair
    hipError_t err;                                         // first event-creation failure
};
extern thread_local LaunchTimer* t_timer;

template <typename F, typename... Args>
inline void launch_kernel(F kernel, dim3 grid, dim3 block, unsigned shmem, hipStream_t s, Args... args) {
    LaunchTimer* t = t_timer;
    if (t && t->err == hipSuccess) {
        auto& pool = *t->pool;
        if (*t->next == pool.size()) {
            hipEvent_t a = nullptr, b = nullptr;
            hipError_t e = hipEventCreate(&a);
            if (e == hipSuccess) e = hipEventCreate(&b);
            if (e != hipSuccess) {
                if (a) (void)hipEventDestroy(a);
                t->err = e;
                hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
                return;
            }
            pool.emplace_back(a, b);
        }
        const auto ev = pool[(*t->next)++];
        hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, ev.first, ev.second, 0u, args...);
        return;
    }
    hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
}

// ---------------------------------------------------------------------------
// Kernel launch parameters
// ---------------------------------------------------------------------------

// Unsigned division by a fixed divisor d >= 1 of numerators below 2^31:
// q = (umulhi(n, mul) + n) >> shift, with shift = ceil(log2 d) and
// mul = floor(2^32 * (2^shift - d) / d) + 1 (round-up multiplier method).
struct FastDiv {
    unsigned mul = 0, shift = 0;
    FastDiv() = default;
    explicit FastDiv(unsigned d) {
        unsigned l = 0;
        while ((1ull << l) < d) ++l;
        shift = l;
        mul = static_cast<unsigned>(((1ull << 32) * ((1ull << l) - d)) / d + 1);
    }
    __host__ __device__ unsigned div(unsigned n) const {
        return static_cast<unsigned>(((static_cast<unsigned long long>(n) * mul >> 32) + n) >> shift);
    }
};

// C[m, n] = act(sum_k A[m, k] * B[n, k] + bias[n] + res[m, n]) for the column
// range of each sub-slice.  A is either a dense row-major matrix or the
// implicit im2col view of an NHWC image (conv).  B is [N][K] row-major.
struct GemmParams {
    const void* A;
    int64_t lda;            // dense A row stride, elements
    // implicit-conv view of A (conv != 0)
    int conv;
    int img_h, img_w, cs;   // input H, W and channel storage stride
    int out_h, out_w;       // output H, W
    int kh, kw, stride, pad;
    FastDiv div_hw, div_w;  // conv: divide by out_h * out_w and by out_w (set by launch_gemm)
    FastDiv div_cs, div_kw; // conv: divide by cs and by kw (set by launch_gemm)
    int dqr, dqc, dc;       // conv: one k sub-stage = (dqr * kw + dqc) taps and dc channels
    const void* B;          // [N][K]
    uint32_t a_bytes, b_bytes;   // extent of A (the whole image for conv) and B (set by launch_gemm)
    const void* bias;       // [N] or null
    const void* res;        // [M][ldc] or null
    void* C;
    int64_t ldc;
    int64_t M;
    int N, K;
    int act;
    int ksub;               // number of sub-slices (decoded from the block index)
    const void* bias2;      // optional second bias [N]
    int out_f32;            // store C as float32 instead of the model dtype
    int epi;                // EPI_STD or EPI_LSTM
    int thin;               // a boundary codec layer: few output columns or a short K, bandwidth-bound
    // EPI_LSTM: columns 4u..4u+3 are gates i, f, g, o of hidden unit u.
    const float* gx;        // [M][ldgx] float32 gate pre-activations added to the product
    int64_t ldgx;
    float* cstate;          // [M][N/4] float32 cell state, read then overwritten
    // the new hidden state of unit u goes to C[m * ldc + u]
    int splits;             // split-K factor (>= 1); > 1 needs `partial`
    float* partial;         // [splits][M][N] float32 partial sums (split-K only)
    // launch geometry, set by the tile launcher: m / n tiles, blocks in all and per XCD,
    // columns (split, sub-slice, n tile) of an m tile, k sub-stages, sub-slice width q and
    // remainder rr, and divisors for the block-index decode
    int g_mt, g_nt, g_total, g_per_xcd, g_cols, g_nk, g_q, g_rr;
    FastDiv g_div_group, g_div_last, g_div_nt, g_div_ksub, g_div_splits;
    FastDiv r_div_groups;   // split-K reduce: divide by ceil(N / 4) (set by launch_gemm)
    // patch-staged 3x3 conv: spatial tiles per image and per tile row, and their divisors
    int h_tiles, h_tx;
    FastDiv h_div_tiles, h_div_tx;
    // 256 x 256 tiles: kWideCtrBytes of tile counters (optional; with them the launch is
    // persistent), and the output span in bytes (set by the launcher)
    unsigned* wide_ctr;
    uint32_t c_bytes;
};
constexpr size_t kWideCtrBytes = 256;

// Split-K factor used for an (M, N, K) product.  A function of the shape
// only -- never of the sub-slice count -- so sub-sliced launches reduce in
// the same order as the unsplit one.
int gemm_splits(int64_t M, int N, int K, int dtype, int epi);
inline size_t gemm_partial_bytes(int64_t M, int N, int splits) {
    return splits > 1 ? static_cast<size_t>(splits) * static_cast<size_t>(M) * static_cast<size_t>(N) * 4 : 0;
}

enum { EPI_STD = 0, EPI_LSTM = 1 };

// Whether a conv runs on the patch-staged 3x3 kernel (bf16, 3x3, stride 1, padding 1, a multiple
// of 64 up to 512 input channels, at most 512 outputs, output from 7 x 7 up to 56 x 56 pixels, at
// most 2^31 multiply-adds over the m output pixels of the batch).  A function of the op's
// geometry only -- never of the sub-slice count -- so sub-sliced and unsplit launches of one op
// take the same path; such convs never split K.
bool conv_halo_ok(int dtype, int kh, int kw, int stride, int pad, int cs, int n_out, int out_h, int out_w,
                  int64_t m);

hipError_t launch_gemm(const GemmParams& p, int dtype, hipStream_t stream);

// The GEMM reads its operands through buffer resources with 32-bit offsets and uses offset
// 2^31 as its out-of-range marker: A (the whole image for a conv) and B must stay below it.
inline bool gemm_operands_fit(int64_t a_bytes, int64_t b_bytes) {
    return a_bytes < (int64_t(1) << 31) && b_bytes < (int64_t(1) << 31);
}

// NCHW float32 -> NHWC (model dtype), channels padded with zeros to cs.
hipError_t launch_nchw_to_nhwc(const float* x, void* y, int n, int c, int h, int w, int cs, int dtype,
                               hipStream_t s);
hipError_t launch_maxpool(const void* x, void* y, int n, int h, int w, int c, int k, int stride, int pad,
                          int ho, int wo, int dtype, hipStream_t s);
hipError_t launch_avgpool(const void* x, void* y, int n, int hw, int c, int dtype, hipStream_t s);
hipError_t launch_layernorm(const void* x, const void* res, const void* g, const void* b, void* y,
                            int64_t rows, int f, float eps, int dtype, hipStream_t s);
// (embeddings clamp ids to [0, vocab): an out-of-range id reads the nearest row, never memory
// past the table)
hipError_t launch_embed_bert(const int32_t* ids, const void* tok, const void* pos, const void* type,
                             const void* g, const void* b, void* y, int batch, int seq, int vocab, int f,
                             float eps, int dtype, hipStream_t s);
hipError_t launch_embed(const int32_t* ids, const void* table, void* y, int64_t n, int f, int vocab, int dtype,
                        hipStream_t s);
hipError_t launch_attention(const void* qkv, void* y, int batch, int seq, int heads, float scale, int dtype,
                            hipStream_t s);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);
// every byte of [p, p + bytes) set to `value` (a fill kernel: safe to record in a graph)
hipError_t launch_fill_bytes(void* p, size_t bytes, unsigned char value, hipStream_t s);
// LSTM recurrence of one layer in a single launch (bf16, hidden a multiple of 16 and at most 1024,
// hidden states and cell state under 2 GiB): hseq[b][t] = h_t from gx = x W_ih^T + b_ih + b_hh
// (float32 [B*T][4H], rows interleaved by unit as the weights).  `sync` holds
// lstm_recurrence_sync_bytes of tile claims, zeroed by the launcher, which also fills hseq
// with 0xFF bytes (the kernel's "not yet stored" mark); cst is scratch for the cell state.
bool lstm_recurrence_ok(int dtype, int64_t batch, int64_t steps, int64_t hidden);
size_t lstm_recurrence_sync_bytes(int64_t batch, int64_t steps, int64_t hidden);
hipError_t launch_lstm_recurrence(const float* gx, const void* whh, void* hseq, float* cst, void* sync, int batch,
                                  int steps, int hidden, hipStream_t s);
// One codec layer y[p][o] = b[o] + sum_c w[o][c] x[p][c] on the vector ALUs, for input widths off
// the GEMM's 16-byte granule; positions * cout < 2^31.
hipError_t launch_codec_narrow(const void* x, const void* w, const void* b, void* y, int64_t positions, int cin,
                               int cout, int dtype, hipStream_t s);
hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t s);

size_t dtype_size(int dtype);

}  // namespace mopar
