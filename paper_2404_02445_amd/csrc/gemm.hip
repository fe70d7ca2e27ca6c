// MFMA GEMM for gfx950: the resource-dominant operators (conv as implicit GEMM
// over NHWC activations, linear layers), the boundary autoencoder and the
// LSTM recurrence all run through this kernel.
//
//   C[m, n] = epilogue( sum_k A[m, k] * B[n, k] )
//
// A is [M][K]: either a dense row-major matrix or the im2col view of an NHWC
// image (k runs over (r, s, c) with c fastest).  B is [N][K] row-major.
//
// Horizontal sub-slicing (the k equal-size sub-slices of an RD operator):
// blockIdx.z selects the sub-slice, whose output columns [lo, hi) and weight
// rows [lo, hi) follow the same split as mopar_subslice_range; each sub-slice
// is tiled on its own and masked at hi.  The K loop -- stage depth, MFMA
// shape, chunk order -- depends only on K and the dtype, never on the tile
// shape or the sub-slice, so every output element goes through the same
// sequence of fp32 operations whatever k is: sub-sliced output equals the
// unsplit output bit for bit.
//
// Data path: each thread streams 16-byte chunks of A and B rows from HBM into
// registers one stage ahead, parks them in LDS (double buffered, rows padded
// by one chunk so the 16 lanes of an MFMA fragment read hit distinct banks),
// and four waves run v_mfma_f32_16x16x32_bf16 (bf16) or
// v_mfma_f32_16x16x4_f32 (fp32) on their wave tile.  The MFMA is issued with
// the weight fragment as the first operand, so each lane ends up holding four
// consecutive output columns of one row: bias, residual, activation, the LSTM
// cell and the store all work on 4-wide vectors.
#include "internal.h"

namespace mopar {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <typename T> struct Elt;
template <> struct Elt<__bf16> { static constexpr int EPC = 8; };   // elements per 16-byte chunk
template <> struct Elt<float> { static constexpr int EPC = 4; };

constexpr int CH = 8;          // 16-byte chunks of each row per LDS stage (128 bytes)
constexpr int RS = CH + 1;     // LDS row stride in chunks (one chunk of padding)

__device__ __forceinline__ float ld_f(const __bf16* p, int64_t i) {
    unsigned short u = reinterpret_cast<const unsigned short*>(p)[i];
    return __uint_as_float(static_cast<unsigned>(u) << 16);
}
__device__ __forceinline__ float ld_f(const float* p, int64_t i) { return p[i]; }

__device__ __forceinline__ float sigmoidf_(float v) { return 1.0f / (1.0f + __expf(-v)); }

__device__ __forceinline__ float act_f(float v, int act) {
    if (act == MOPAR_ACT_RELU) return v > 0.0f ? v : 0.0f;
    if (act == MOPAR_ACT_GELU) return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
    return v;
}

template <typename T>
__device__ __forceinline__ void store4(T* c, int64_t idx, const float* v, int nvalid, bool vec_ok);

template <>
__device__ __forceinline__ void store4<__bf16>(__bf16* c, int64_t idx, const float* v, int nvalid, bool vec_ok) {
    if (nvalid == 4 && vec_ok) {
        typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
        bf16x4 o = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
        *reinterpret_cast<bf16x4*>(c + idx) = o;
    } else {
        for (int i = 0; i < nvalid; ++i) c[idx + i] = (__bf16)v[i];
    }
}

template <>
__device__ __forceinline__ void store4<float>(float* c, int64_t idx, const float* v, int nvalid, bool vec_ok) {
    if (nvalid == 4 && vec_ok) {
        *reinterpret_cast<f32x4*>(c + idx) = f32x4{v[0], v[1], v[2], v[3]};
    } else {
        for (int i = 0; i < nvalid; ++i) c[idx + i] = v[i];
    }
}

template <typename T, int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256) void gemm_kernel(const GemmParams p) {
    constexpr int EPC = Elt<T>::EPC;
    constexpr int BK = CH * EPC;              // K elements per stage
    constexpr int TM = BM / WM, TN = BN / WN; // wave tile
    constexpr int FM = TM / 16, FN = TN / 16; // 16x16 MFMA tiles per wave
    constexpr int NCHUNK = (BM + BN) * CH;
    constexpr int PER = (NCHUNK + 255) / 256;
    static_assert(WM * WN == 4 && FM >= 1 && FN >= 1, "tile");

    __shared__ uint4 lds[2][(BM + BN) * RS];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;

    // sub-slice j owns columns [n_lo, n_hi)
    const int j = blockIdx.z;
    const int q = p.N / p.ksub, rr = p.N % p.ksub;
    const int n_lo = j * q + min(j, rr), n_hi = (j + 1) * q + min(j + 1, rr);
    const int n0 = n_lo + blockIdx.y * BN;
    if (n0 >= n_hi) return;                   // block-uniform: this tile lies past the sub-slice
    const int64_t m0 = static_cast<int64_t>(blockIdx.x) * BM;

    const T* __restrict__ Ap = static_cast<const T*>(p.A);
    const T* __restrict__ Bp = static_cast<const T*>(p.B);

    // --- per-thread load assignment: chunk column fixed, PER rows ---------------------
    const int col = tid % CH;
    const T* rowptr[PER];        // dense A / B: row base; conv A: image base
    int hb[PER], wb[PER];        // conv A: top-left input coordinate of the row's window
    bool rvalid[PER];
    bool is_a[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int row = tid / CH + i * (256 / CH);
        rvalid[i] = false;
        is_a[i] = row < BM;
        rowptr[i] = nullptr;
        hb[i] = wb[i] = 0;
        if (row >= BM + BN) continue;
        if (row < BM) {
            const int64_t m = m0 + row;
            if (m >= p.M) continue;
            rvalid[i] = true;
            if (p.conv) {
                const int64_t hw = static_cast<int64_t>(p.out_h) * p.out_w;
                const int64_t img = m / hw;
                const int rem = static_cast<int>(m - img * hw);
                const int ho = rem / p.out_w, wo = rem - (rem / p.out_w) * p.out_w;
                rowptr[i] = Ap + img * p.img_h * p.img_w * static_cast<int64_t>(p.cs);
                hb[i] = ho * p.stride - p.pad;
                wb[i] = wo * p.stride - p.pad;
            } else {
                rowptr[i] = Ap + m * p.lda;
            }
        } else {
            const int n = n0 + (row - BM);
            if (n >= n_hi) continue;
            rvalid[i] = true;
            rowptr[i] = Bp + static_cast<int64_t>(n) * p.K;
        }
    }

    uint4 stage[PER];
    auto load_stage = [&](int kt) {
        const int k = kt * BK + col * EPC;
        const bool kin = k < p.K;
        // conv: decompose k -> (tap row rr, tap col ss, channel ci); one chunk never
        // straddles taps because cs is a multiple of EPC
        int dr = 0, ds = 0, ci = 0;
        if (p.conv && kin) {
            const int tap = k / p.cs;
            ci = k - tap * p.cs;
            dr = tap / p.kw;
            ds = tap - dr * p.kw;
        }
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            uint4 v = make_uint4(0, 0, 0, 0);
            if (rvalid[i] && kin) {
                if (is_a[i] && p.conv) {
                    const int hi = hb[i] + dr, wi = wb[i] + ds;
                    if (hi >= 0 && hi < p.img_h && wi >= 0 && wi < p.img_w)
                        v = *reinterpret_cast<const uint4*>(
                            rowptr[i] + (static_cast<int64_t>(hi) * p.img_w + wi) * p.cs + ci);
                } else {
                    v = *reinterpret_cast<const uint4*>(rowptr[i] + k);
                }
            }
            stage[i] = v;
        }
    };
    auto store_stage = [&](int buf) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int row = tid / CH + i * (256 / CH);
            if (row < BM + BN) lds[buf][row * RS + col] = stage[i];
        }
    };

    f32x4 acc[FM][FN];
#pragma unroll
    for (int a = 0; a < FM; ++a)
#pragma unroll
        for (int b = 0; b < FN; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk = (p.K + BK - 1) / BK;
    load_stage(0);
    store_stage(0);
    __syncthreads();

    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) load_stage(kt + 1);
        const uint4* L = lds[buf];
#pragma unroll
        for (int ks = 0; ks < CH / 4; ++ks) {
            const int chunk = ks * 4 + (lane >> 4);
            uint4 af[FM], bf[FN];
#pragma unroll
            for (int a = 0; a < FM; ++a) af[a] = L[(wm * TM + a * 16 + (lane & 15)) * RS + chunk];
#pragma unroll
            for (int b = 0; b < FN; ++b) bf[b] = L[(BM + wn * TN + b * 16 + (lane & 15)) * RS + chunk];
#pragma unroll
            for (int a = 0; a < FM; ++a)
#pragma unroll
                for (int b = 0; b < FN; ++b) {
                    if constexpr (sizeof(T) == 2) {
                        acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            __builtin_bit_cast(bf16x8, bf[b]), __builtin_bit_cast(bf16x8, af[a]), acc[a][b], 0, 0, 0);
                    } else {
                        const f32x4 av = __builtin_bit_cast(f32x4, af[a]);
                        const f32x4 bv = __builtin_bit_cast(f32x4, bf[b]);
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(bv[e], av[e], acc[a][b], 0, 0, 0);
                    }
                }
        }
        if (kt + 1 < nk) store_stage(buf ^ 1);
        __syncthreads();
    }

    // --- epilogue: lane holds rows m, columns n..n+3 --------------------------------------
    const T* bias = static_cast<const T*>(p.bias);
    const T* bias2 = static_cast<const T*>(p.bias2);
    const T* res = static_cast<const T*>(p.res);
#pragma unroll
    for (int a = 0; a < FM; ++a) {
        const int64_t m = m0 + wm * TM + a * 16 + (lane & 15);
        if (m >= p.M) continue;
#pragma unroll
        for (int b = 0; b < FN; ++b) {
            const int n = n0 + wn * TN + b * 16 + (lane >> 4) * 4;
            if (n >= n_hi) continue;
            const int nvalid = min(4, n_hi - n);
            float v[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = acc[a][b][i];
            if (p.epi == EPI_LSTM) {
                // gates i, f, g, o of unit n / 4 (n is a multiple of 4 and nvalid == 4)
                const f32x4 g4 = *reinterpret_cast<const f32x4*>(p.gx + m * p.ldgx + n);
                const float gi = v[0] + g4[0], gf = v[1] + g4[1], gg = v[2] + g4[2], go = v[3] + g4[3];
                const int u = n >> 2;
                float* cp = p.cstate + m * (p.N >> 2) + u;
                const float c = sigmoidf_(gf) * *cp + sigmoidf_(gi) * tanhf(gg);
                *cp = c;
                const float h = sigmoidf_(go) * tanhf(c);
                static_cast<T*>(p.C)[m * p.ldc + u] = static_cast<T>(h);
                continue;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (i < nvalid) {
                    if (bias) v[i] += ld_f(bias, n + i);
                    if (bias2) v[i] += ld_f(bias2, n + i);
                    if (res) v[i] += ld_f(res, m * p.ldc + n + i);
                    v[i] = act_f(v[i], p.act);
                }
            }
            const int64_t idx = m * p.ldc + n;
            if (p.out_f32)
                store4<float>(static_cast<float*>(p.C), idx, v, nvalid, (idx & 3) == 0);
            else
                store4<T>(static_cast<T*>(p.C), idx, v, nvalid, (idx & 3) == 0);
        }
    }
}

// ---------------------------------------------------------------------------
// Tile selection.  All shapes share the K loop, so the choice only affects
// speed, never the bits of the result.
// ---------------------------------------------------------------------------

template <typename T, int BM, int BN, int WM, int WN>
static hipError_t launch_cfg(const GemmParams& p, int width, hipStream_t s) {
    dim3 grid(static_cast<unsigned>((p.M + BM - 1) / BM), static_cast<unsigned>((width + BN - 1) / BN),
              static_cast<unsigned>(p.ksub));
    hipLaunchKernelGGL((gemm_kernel<T, BM, BN, WM, WN>), grid, dim3(256), 0, s, p);
    return hipGetLastError();
}

template <typename T>
static hipError_t dispatch(const GemmParams& p, hipStream_t s) {
    const int width = (p.N + p.ksub - 1) / p.ksub;   // widest sub-slice
    if (p.epi == EPI_LSTM || p.M <= 64) {
        if (p.M <= 16) return launch_cfg<T, 16, 64, 1, 4>(p, width, s);
        if (width >= 64 && p.epi != EPI_LSTM) return launch_cfg<T, 64, 64, 2, 2>(p, width, s);
        return launch_cfg<T, 64, 16, 4, 1>(p, width, s);
    }
    const int64_t mt = (p.M + 127) / 128;
    auto blocks = [&](int bn) { return mt * ((width + bn - 1) / bn) * p.ksub; };
    if (width >= 128 && blocks(128) >= 512) return launch_cfg<T, 128, 128, 2, 2>(p, width, s);
    if (width >= 64 && blocks(64) >= 256) return launch_cfg<T, 128, 64, 2, 2>(p, width, s);
    if (width >= 32) return launch_cfg<T, 128, 32, 4, 1>(p, width, s);
    return launch_cfg<T, 128, 16, 4, 1>(p, width, s);
}

hipError_t launch_gemm(const GemmParams& p, int dtype, hipStream_t stream) {
    if (p.M <= 0 || p.N <= 0) return hipSuccess;
    if (dtype == MOPAR_BF16) return dispatch<__bf16>(p, stream);
    return dispatch<float>(p, stream);
}

}  // namespace mopar
