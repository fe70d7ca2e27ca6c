// Bandwidth-bound kernels of the sliced forward pass (gfx950, wave64):
// input layout conversion, pooling, layer norm, embeddings, attention and the
// raw boundary copy.  Accesses are 16-byte vectors along the contiguous
// (channel / feature) dimension wherever the shape allows; reductions are
// wave-level butterflies (no atomics, so results are reproducible).
#include "internal.h"

namespace mopar {

template <typename T> struct Vec;   // 16-byte vector of T
template <> struct Vec<__bf16> { static constexpr int N = 8; };
template <> struct Vec<float> { static constexpr int N = 4; };

__device__ __forceinline__ float to_f(__bf16 v) {
    return __uint_as_float(static_cast<unsigned>(__builtin_bit_cast(unsigned short, v)) << 16);
}
__device__ __forceinline__ float to_f(float v) { return v; }

template <typename T> __device__ __forceinline__ T from_f(float v) { return static_cast<T>(v); }

// Sum over the wave, the same value in every lane: within each row of 16 lanes a butterfly of
// DPP moves (partners 1 and 2 apart, then the mirrored half, then the mirrored row: each step
// adds a lane's partial to its partner's, so all lanes of a row agree), then the four row sums
// are read out and added in row order.
__device__ __forceinline__ float dpp_add(float v, int ctrl_sel) {
    int m = 0;
    switch (ctrl_sel) {   // DPP controls must be compile-time constants
        case 0: m = __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false); break;   // quad [1,0,3,2]
        case 1: m = __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false); break;   // quad [2,3,0,1]
        case 2: m = __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false); break;  // row half mirror
        default: m = __builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false); break; // row mirror
    }
    return v + __int_as_float(m);
}
__device__ __forceinline__ float wave_sum(float v) {
    v = dpp_add(v, 0);
    v = dpp_add(v, 1);
    v = dpp_add(v, 2);
    v = dpp_add(v, 3);
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return (r0 + r1) + (r2 + r3);
}

static inline unsigned blocks_for(int64_t n, int per_block) {
    int64_t b = (n + per_block - 1) / per_block;
    return static_cast<unsigned>(b < 1 ? 1 : b);
}

// ---------------------------------------------------------------------------
// NCHW float32 (model input) -> NHWC in the model dtype, channels padded to cs.
// One thread per pixel: C strided reads (coalesced across neighbouring w),
// cs-wide contiguous 16-byte writes.  Sizes below 2^31 elements (host-checked).
// ---------------------------------------------------------------------------
template <typename T>
__global__ void nchw_to_nhwc_kernel(const float* __restrict__ x, T* __restrict__ y, int n, int c, int h, int w,
                                    int cs) {
    constexpr int V = Vec<T>::N;
    const int pix = blockIdx.x * blockDim.x + threadIdx.x;
    const int hw = h * w;
    if (pix >= n * hw) return;
    const int img = pix / hw, r = pix - img * hw;
    const float* src = x + static_cast<int64_t>(img) * c * hw + r;
    T* dst = y + static_cast<int64_t>(pix) * cs;
    for (int c0 = 0; c0 < cs; c0 += V) {           // cs is a multiple of V
        // every channel slot loads (padding slots re-read channel c - 1), so the loads go out
        // together instead of one branch and one wait per channel
        float f[V];
#pragma unroll
        for (int i = 0; i < V; ++i) f[i] = src[static_cast<int64_t>(min(c0 + i, c - 1)) * hw];
        uint4 out;
        T* o = reinterpret_cast<T*>(&out);
#pragma unroll
        for (int i = 0; i < V; ++i) o[i] = from_f<T>(c0 + i < c ? f[i] : 0.0f);
        *reinterpret_cast<uint4*>(dst + c0) = out;
    }
}

hipError_t launch_nchw_to_nhwc(const float* x, void* y, int n, int c, int h, int w, int cs, int dtype,
                               hipStream_t s) {
    const int64_t pix = static_cast<int64_t>(n) * h * w;
    if (pix * cs >= (int64_t(1) << 31) || cs % (dtype == MOPAR_BF16 ? 8 : 4) != 0) return hipErrorInvalidValue;
    if (dtype == MOPAR_BF16)
        launch_kernel(nchw_to_nhwc_kernel<__bf16>, dim3(blocks_for(pix, 256)), dim3(256), 0, s, x,
                           static_cast<__bf16*>(y), n, c, h, w, cs);
    else
        launch_kernel(nchw_to_nhwc_kernel<float>, dim3(blocks_for(pix, 256)), dim3(256), 0, s, x,
                           static_cast<float*>(y), n, c, h, w, cs);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Max pool, NHWC: one thread per (output pixel, 16-byte channel group).
// Window positions outside the image count as -inf.  KW > 0 fixes the window
// size at compile time; every position then loads (an outside one re-reads a
// clamped pixel and is ignored), so all the window's loads issue together.
// Sizes below 2^31 elements (host-checked): 32-bit index math.
// ---------------------------------------------------------------------------
template <typename T, int KW>
__global__ void maxpool_kernel(const T* __restrict__ x, T* __restrict__ y, int n, int h, int w, int c, int kr,
                               int stride, int pad, int ho, int wo) {
    constexpr int V = Vec<T>::N;
    const int k = KW > 0 ? KW : kr;
    const int groups = c / V;
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n * ho * wo * groups) return;
    const int pix = t / groups, g = t - pix * groups;
    const int img = pix / (ho * wo), rem = pix - img * (ho * wo);
    const int oy = rem / wo, ox = rem - oy * wo;
    float m[V];
#pragma unroll
    for (int i = 0; i < V; ++i) m[i] = -INFINITY;
    if constexpr (KW > 0) {
        uint4 raw[KW * KW];
#pragma unroll
        for (int r = 0; r < KW; ++r)
#pragma unroll
            for (int q = 0; q < KW; ++q) {
                const int iy = min(max(oy * stride - pad + r, 0), h - 1);
                const int ix = min(max(ox * stride - pad + q, 0), w - 1);
                raw[r * KW + q] = *reinterpret_cast<const uint4*>(x + ((img * h + iy) * w + ix) * c + g * V);
            }
#pragma unroll
        for (int r = 0; r < KW; ++r)
#pragma unroll
            for (int q = 0; q < KW; ++q) {
                const int iy = oy * stride - pad + r, ix = ox * stride - pad + q;
                const bool in = static_cast<unsigned>(iy) < static_cast<unsigned>(h) &&
                                static_cast<unsigned>(ix) < static_cast<unsigned>(w);
                const T* e = reinterpret_cast<const T*>(&raw[r * KW + q]);
#pragma unroll
                for (int i = 0; i < V; ++i) m[i] = fmaxf(m[i], in ? to_f(e[i]) : -INFINITY);
            }
    } else {
        for (int r = 0; r < k; ++r) {
            const int iy = oy * stride - pad + r;
            for (int q = 0; q < k; ++q) {
                const int ix = ox * stride - pad + q;
                if (static_cast<unsigned>(iy) >= static_cast<unsigned>(h) ||
                    static_cast<unsigned>(ix) >= static_cast<unsigned>(w))
                    continue;
                const uint4 raw = *reinterpret_cast<const uint4*>(x + ((img * h + iy) * w + ix) * c + g * V);
                const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
                for (int i = 0; i < V; ++i) m[i] = fmaxf(m[i], to_f(e[i]));
            }
        }
    }
    uint4 out;
    T* o = reinterpret_cast<T*>(&out);
#pragma unroll
    for (int i = 0; i < V; ++i) o[i] = from_f<T>(m[i]);
    *reinterpret_cast<uint4*>(y + pix * c + g * V) = out;
}

template <typename T>
static void maxpool_launch(const void* x, void* y, int n, int h, int w, int c, int k, int stride, int pad, int ho,
                           int wo, hipStream_t s) {
    const int64_t total = static_cast<int64_t>(n) * ho * wo * (c / Vec<T>::N);
    const T* xp = static_cast<const T*>(x);
    T* yp = static_cast<T*>(y);
    if (k == 3)
        launch_kernel((maxpool_kernel<T, 3>), dim3(blocks_for(total, 256)), dim3(256), 0, s, xp, yp, n, h, w, c, k,
                           stride, pad, ho, wo);
    else if (k == 2)
        launch_kernel((maxpool_kernel<T, 2>), dim3(blocks_for(total, 256)), dim3(256), 0, s, xp, yp, n, h, w, c, k,
                           stride, pad, ho, wo);
    else
        launch_kernel((maxpool_kernel<T, 0>), dim3(blocks_for(total, 256)), dim3(256), 0, s, xp, yp, n, h, w, c, k,
                           stride, pad, ho, wo);
}

hipError_t launch_maxpool(const void* x, void* y, int n, int h, int w, int c, int k, int stride, int pad, int ho,
                          int wo, int dtype, hipStream_t s) {
    if (static_cast<int64_t>(n) * h * w * c >= (int64_t(1) << 31)) return hipErrorInvalidValue;
    // the kernel moves whole 16-byte channel groups: a channel count off the granule is refused
    if (c % (dtype == MOPAR_BF16 ? 8 : 4) != 0) return hipErrorInvalidValue;
    if (dtype == MOPAR_BF16)
        maxpool_launch<__bf16>(x, y, n, h, w, c, k, stride, pad, ho, wo, s);
    else
        maxpool_launch<float>(x, y, n, h, w, c, k, stride, pad, ho, wo, s);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Global average pool, NHWC -> [N][C].  A block owns one image and 8 channel
// chunks (16 bytes each); its 256 threads are 8 chunks x 32 pixel slices.
// Slice s sums pixels s, s + 32, ... in order (fp32); the 32 slice sums are
// then added in slice order and divided once: a fixed order, so the result
// is reproducible.  Channel counts that are not a whole number of chunks use
// one thread per channel, summing pixels in order.
// ---------------------------------------------------------------------------
constexpr int AP_SLICES = 32, AP_CHUNKS = 8;

template <typename T>
__global__ __launch_bounds__(256) void avgpool_kernel(const T* __restrict__ x, T* __restrict__ y, int hw, int c) {
    constexpr int V = Vec<T>::N;
    __shared__ float part[AP_SLICES][AP_CHUNKS * V];
    const int img = blockIdx.y;
    const int chunk = threadIdx.x % AP_CHUNKS, slice = threadIdx.x / AP_CHUNKS;
    const int c0 = (blockIdx.x * AP_CHUNKS + chunk) * V;
    float sum[V];
#pragma unroll
    for (int i = 0; i < V; ++i) sum[i] = 0.0f;
    if (c0 < c) {
        const T* p = x + static_cast<int64_t>(img) * hw * c + c0;
        for (int px = slice; px < hw; px += AP_SLICES) {
            const uint4 raw = *reinterpret_cast<const uint4*>(p + static_cast<int64_t>(px) * c);
            const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
            for (int i = 0; i < V; ++i) sum[i] += to_f(e[i]);
        }
    }
#pragma unroll
    for (int i = 0; i < V; ++i) part[slice][chunk * V + i] = sum[i];
    __syncthreads();
    if (threadIdx.x < AP_CHUNKS * V) {
        const int ch = blockIdx.x * AP_CHUNKS * V + threadIdx.x;
        if (ch < c) {
            float s = 0.0f;
            for (int sl = 0; sl < AP_SLICES; ++sl) s += part[sl][threadIdx.x];
            y[static_cast<int64_t>(img) * c + ch] = from_f<T>(s / static_cast<float>(hw));
        }
    }
}

template <typename T>
__global__ void avgpool_channel_kernel(const T* __restrict__ x, T* __restrict__ y, int n, int hw, int c) {
    const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (t >= static_cast<int64_t>(n) * c) return;
    const int64_t img = t / c;
    const int ch = static_cast<int>(t - img * c);
    const T* p = x + img * hw * c + ch;
    float s = 0.0f;
    for (int i = 0; i < hw; ++i) s += to_f(p[static_cast<int64_t>(i) * c]);
    y[t] = from_f<T>(s / static_cast<float>(hw));
}

template <typename T>
static void avgpool_launch(const void* x, void* y, int n, int hw, int c, hipStream_t s) {
    constexpr int V = Vec<T>::N;
    if (c % V == 0) {
        const dim3 grid((c / V + AP_CHUNKS - 1) / AP_CHUNKS, n);
        launch_kernel(avgpool_kernel<T>, grid, dim3(256), 0, s, static_cast<const T*>(x), static_cast<T*>(y), hw, c);
    } else {
        launch_kernel(avgpool_channel_kernel<T>, dim3(blocks_for(static_cast<int64_t>(n) * c, 256)), dim3(256), 0, s,
                           static_cast<const T*>(x), static_cast<T*>(y), n, hw, c);
    }
}

hipError_t launch_avgpool(const void* x, void* y, int n, int hw, int c, int dtype, hipStream_t s) {
    if (dtype == MOPAR_BF16)
        avgpool_launch<__bf16>(x, y, n, hw, c, s);
    else
        avgpool_launch<float>(x, y, n, hw, c, s);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Layer norm over rows of F <= 64 * LN_MAXV elements: one wave per row, the
// row held in registers, mean then centred variance by wave butterflies.
// When F is a whole number of 16-byte chunks each lane holds whole chunks
// (chunk lane + 64 j), read and written as vectors, and the kernel instance
// keeps MV floats per lane -- just the row's chunks, so fewer registers and
// more resident waves; otherwise element lane + 64 i, MV = LN_MAXV.
// ---------------------------------------------------------------------------
constexpr int LN_MAXV = 32;

// column of register i of this lane
template <typename T, bool VEC>
__device__ __forceinline__ int ln_col(int lane, int i) {
    constexpr int V = Vec<T>::N;
    return VEC ? (lane + 64 * (i / V)) * V + i % V : lane + 64 * i;
}

template <typename T, bool VEC, int MV>
__device__ __forceinline__ void ln_row(float (&v)[MV], int f, int lane, const T* g, const T* b, float eps,
                                       T* out) {
    constexpr int V = Vec<T>::N;
    // gamma and beta go out before the reductions, so their latency overlaps the row's
    uint4 gr[VEC ? MV / V : 1], br[VEC ? MV / V : 1];
    if constexpr (VEC) {
#pragma unroll
        for (int j = 0; j < MV / V; ++j) {
            const int c0 = min((lane + 64 * j) * V, f - V);   // in range; unused past f
            gr[j] = *reinterpret_cast<const uint4*>(g + c0);
            br[j] = *reinterpret_cast<const uint4*>(b + c0);
        }
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < MV; ++i)
        if (ln_col<T, VEC>(lane, i) < f) s += v[i];
    const float mean = wave_sum(s) / static_cast<float>(f);
    float q = 0.0f;
#pragma unroll
    for (int i = 0; i < MV; ++i)
        if (ln_col<T, VEC>(lane, i) < f) {
            const float d = v[i] - mean;
            q += d * d;
        }
    const float var = wave_sum(q) / static_cast<float>(f);
    const float inv = 1.0f / sqrtf(var + eps);
    if constexpr (VEC) {
#pragma unroll
        for (int j = 0; j < MV / V; ++j) {
            const int c0 = (lane + 64 * j) * V;
            if (c0 >= f) continue;
            const T* ge = reinterpret_cast<const T*>(&gr[j]);
            const T* be = reinterpret_cast<const T*>(&br[j]);
            uint4 o;
            T* oe = reinterpret_cast<T*>(&o);
#pragma unroll
            for (int e = 0; e < V; ++e) oe[e] = from_f<T>((v[j * V + e] - mean) * inv * to_f(ge[e]) + to_f(be[e]));
            *reinterpret_cast<uint4*>(out + c0) = o;
        }
    } else {
#pragma unroll
        for (int i = 0; i < MV; ++i) {
            const int col = lane + i * 64;
            if (col < f) out[col] = from_f<T>((v[i] - mean) * inv * to_f(g[col]) + to_f(b[col]));
        }
    }
}

// v[i] = a[col] (+ c[col]) for this lane's columns (zeros past f)
template <typename T, bool VEC, int MV>
__device__ __forceinline__ void ln_load(const T* a, const T* c, int f, int lane, float (&v)[MV]) {
    constexpr int V = Vec<T>::N;
    if constexpr (VEC) {
        // Every lane loads (a lane past f re-reads the last chunk and keeps zeros): per-lane
        // branches around the loads would make each chunk wait for the previous one.
        uint4 ar[MV / V], cr[MV / V];
#pragma unroll
        for (int j = 0; j < MV / V; ++j) {
            const int cc = min((lane + 64 * j) * V, f - V);
            ar[j] = *reinterpret_cast<const uint4*>(a + cc);
            cr[j] = c ? *reinterpret_cast<const uint4*>(c + cc) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < MV / V; ++j) {
            const bool ok = (lane + 64 * j) * V < f;
            const T* ae = reinterpret_cast<const T*>(&ar[j]);
            const T* ce = reinterpret_cast<const T*>(&cr[j]);
#pragma unroll
            for (int e = 0; e < V; ++e) v[j * V + e] = ok ? to_f(ae[e]) + (c ? to_f(ce[e]) : 0.0f) : 0.0f;
        }
    } else {
#pragma unroll
        for (int i = 0; i < MV; ++i) {
            const int col = lane + i * 64;
            v[i] = col < f ? to_f(a[col]) + (c ? to_f(c[col]) : 0.0f) : 0.0f;
        }
    }
}

template <typename T, bool VEC, int MV>
__global__ void layernorm_kernel(const T* __restrict__ x, const T* __restrict__ res, const T* __restrict__ g,
                                 const T* __restrict__ b, T* __restrict__ y, int64_t rows, int f, float eps) {
    const int lane = threadIdx.x & 63;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * (blockDim.x / 64) + (threadIdx.x >> 6);
    if (row >= rows) return;
    float v[MV];
    ln_load<T, VEC, MV>(x + row * f, res ? res + row * f : nullptr, f, lane, v);
    ln_row<T, VEC, MV>(v, f, lane, g, b, eps, y + row * f);
}

// go(kernel) with the row kernel instance for f columns: 16-byte chunks when f allows, with as
// many per lane as the row needs (fewer registers, more resident waves), else one element
// per lane and step
template <typename T, template <typename, bool, int> class K, typename Go>
static void ln_instance(int f, Go&& go) {
    constexpr int V = Vec<T>::N;
    if (f % V != 0) return go(K<T, false, LN_MAXV>::fn);
    switch ((f + 64 * V - 1) / (64 * V)) {
        case 1: return go(K<T, true, V>::fn);
        case 2: return go(K<T, true, 2 * V>::fn);
        case 3: return go(K<T, true, 3 * V>::fn);
        case 4: return go(K<T, true, 4 * V>::fn);
        default: return go(K<T, true, LN_MAXV>::fn);
    }
}
template <typename T, bool VEC, int MV>
struct LnK { static constexpr auto fn = layernorm_kernel<T, VEC, MV>; };

template <typename T>
static void layernorm_launch(const void* x, const void* res, const void* g, const void* b, void* y, int64_t rows,
                             int f, float eps, hipStream_t s) {
    const T *xp = static_cast<const T*>(x), *rp = static_cast<const T*>(res);
    const T *gp = static_cast<const T*>(g), *bp = static_cast<const T*>(b);
    ln_instance<T, LnK>(f, [&](auto kern) {
        launch_kernel(kern, dim3(blocks_for(rows, 4)), dim3(256), 0, s, xp, rp, gp, bp, static_cast<T*>(y), rows, f,
                      eps);
    });
}

hipError_t launch_layernorm(const void* x, const void* res, const void* g, const void* b, void* y, int64_t rows,
                            int f, float eps, int dtype, hipStream_t s) {
    if (f < 1 || f > 64 * LN_MAXV) return hipErrorInvalidValue;   // a row lives in one wave's registers
    if (dtype == MOPAR_BF16)
        layernorm_launch<__bf16>(x, res, g, b, y, rows, f, eps, s);
    else
        layernorm_launch<float>(x, res, g, b, y, rows, f, eps, s);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// BERT embedding: v = tok[id] + pos[s] + type[0], then layer norm (one wave
// per token).
// ---------------------------------------------------------------------------
template <typename T, bool VEC, int MV>
__global__ void embed_bert_kernel(const int32_t* __restrict__ ids, const T* __restrict__ tok,
                                  const T* __restrict__ pos, const T* __restrict__ type, const T* __restrict__ g,
                                  const T* __restrict__ b, T* __restrict__ y, int64_t rows, int seq, int vocab, int f,
                                  float eps) {
    const int lane = threadIdx.x & 63;
    const int64_t row = static_cast<int64_t>(blockIdx.x) * (blockDim.x / 64) + (threadIdx.x >> 6);
    if (row >= rows) return;
    const int sidx = static_cast<int>(row % seq);
    const T* tr = tok + static_cast<int64_t>(min(max(ids[row], 0), vocab - 1)) * f;   // ids clamped to the table
    const T* pr = pos + static_cast<int64_t>(sidx) * f;
    float v[MV];
    ln_load<T, VEC, MV>(tr, pr, f, lane, v);
    float t[MV];
    ln_load<T, VEC, MV>(type, nullptr, f, lane, t);
#pragma unroll
    for (int i = 0; i < MV; ++i) v[i] += t[i];
    ln_row<T, VEC, MV>(v, f, lane, g, b, eps, y + row * f);
}

template <typename T, bool VEC, int MV>
struct EmbK { static constexpr auto fn = embed_bert_kernel<T, VEC, MV>; };

template <typename T>
static void embed_bert_launch(const int32_t* ids, const void* tok, const void* pos, const void* type, const void* g,
                              const void* b, void* y, int64_t rows, int seq, int vocab, int f, float eps,
                              hipStream_t s) {
    const T *tp = static_cast<const T*>(tok), *pp = static_cast<const T*>(pos), *yp = static_cast<const T*>(type);
    const T *gp = static_cast<const T*>(g), *bp = static_cast<const T*>(b);
    ln_instance<T, EmbK>(f, [&](auto kern) {
        launch_kernel(kern, dim3(blocks_for(rows, 4)), dim3(256), 0, s, ids, tp, pp, yp, gp, bp, static_cast<T*>(y),
                      rows, seq, vocab, f, eps);
    });
}

hipError_t launch_embed_bert(const int32_t* ids, const void* tok, const void* pos, const void* type, const void* g,
                             const void* b, void* y, int batch, int seq, int vocab, int f, float eps, int dtype,
                             hipStream_t s) {
    const int64_t rows = static_cast<int64_t>(batch) * seq;
    if (vocab < 1 || f < 1 || f > 64 * LN_MAXV) return hipErrorInvalidValue;
    if (dtype == MOPAR_BF16)
        embed_bert_launch<__bf16>(ids, tok, pos, type, g, b, y, rows, seq, vocab, f, eps, s);
    else
        embed_bert_launch<float>(ids, tok, pos, type, g, b, y, rows, seq, vocab, f, eps, s);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Plain embedding gather: one thread per 16-byte chunk of an output row.
// ---------------------------------------------------------------------------
// one block per token: the id is one (scalar) load per block, then the row's 16-byte chunks
// (an id outside [0, vocab) reads the nearest valid row instead of memory past the table)
__global__ __launch_bounds__(128) void embed_kernel(const int32_t* __restrict__ ids, const uint4* __restrict__ table,
                                                    uint4* __restrict__ y, int chunks, int vocab) {
    const int64_t row = blockIdx.x;
    const uint4* src = table + static_cast<int64_t>(min(max(ids[row], 0), vocab - 1)) * chunks;
    uint4* dst = y + row * chunks;
    for (int c = threadIdx.x; c < chunks; c += 128) dst[c] = src[c];
}

hipError_t launch_embed(const int32_t* ids, const void* table, void* y, int64_t n, int f, int vocab, int dtype,
                        hipStream_t s) {
    const int chunks = static_cast<int>(f * dtype_size(dtype) / 16);
    if (n >= (int64_t(1) << 31) || vocab < 1) return hipErrorInvalidValue;
    if (n == 0) return hipSuccess;
    launch_kernel(embed_kernel, dim3(static_cast<unsigned>(n)), dim3(128), 0, s, ids, static_cast<const uint4*>(table),
                  static_cast<uint4*>(y), chunks, vocab);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Multi-head self-attention, head dim 64, seq <= 128.  One block per (b, h):
// K and V of the head staged in LDS as fp32; one thread per query row runs
// the softmax online (running max and normaliser) and accumulates P.V in
// registers.  Scores and probabilities never leave registers.
// ---------------------------------------------------------------------------
constexpr int ATT_D = 64;
constexpr int ATT_MAXS = 128;

template <typename T>
__global__ __launch_bounds__(ATT_MAXS) void attention_kernel(const T* __restrict__ qkv, T* __restrict__ y, int seq,
                                                             int heads, float scale) {
    __shared__ float ks[ATT_MAXS][ATT_D];   // read as broadcasts: no padding needed
    __shared__ float vs[ATT_MAXS][ATT_D];
    const int b = blockIdx.x / heads, h = blockIdx.x % heads;
    const int f = heads * ATT_D;
    const T* base = qkv + static_cast<int64_t>(b) * seq * 3 * f;
    for (int idx = threadIdx.x; idx < seq * ATT_D; idx += blockDim.x) {
        const int r = idx / ATT_D, e = idx % ATT_D;
        ks[r][e] = to_f(base[static_cast<int64_t>(r) * 3 * f + f + h * ATT_D + e]);
        vs[r][e] = to_f(base[static_cast<int64_t>(r) * 3 * f + 2 * f + h * ATT_D + e]);
    }
    __syncthreads();
    const int i = threadIdx.x;
    if (i >= seq) return;
    float q[ATT_D], o[ATT_D];
    const T* qr = base + static_cast<int64_t>(i) * 3 * f + h * ATT_D;
#pragma unroll
    for (int e = 0; e < ATT_D; ++e) {
        q[e] = to_f(qr[e]);
        o[e] = 0.0f;
    }
    float mx = -INFINITY, den = 0.0f;
    for (int jj = 0; jj < seq; ++jj) {
        float sc = 0.0f;
#pragma unroll
        for (int e = 0; e < ATT_D; ++e) sc += q[e] * ks[jj][e];
        sc *= scale;
        const float mnew = fmaxf(mx, sc);
        const float corr = __expf(mx - mnew);
        const float pj = __expf(sc - mnew);
        den = den * corr + pj;
#pragma unroll
        for (int e = 0; e < ATT_D; ++e) o[e] = o[e] * corr + pj * vs[jj][e];
        mx = mnew;
    }
    const float inv = 1.0f / den;
    T* yr = y + (static_cast<int64_t>(b) * seq + i) * f + h * ATT_D;
#pragma unroll
    for (int e = 0; e < ATT_D; ++e) yr[e] = from_f<T>(o[e] * inv);
}

// ---------------------------------------------------------------------------
// bf16 attention on the matrix cores.  One block per (batch, head, 64-query
// tile), four waves of 16 query rows.  Q, K (row-major) and V (transposed,
// [dim][key]) are staged in LDS with padded rows so the 16 lanes of an MFMA
// fragment hit distinct banks.  S = Q K^T accumulates in fp32
// (v_mfma_f32_16x16x32_bf16, key fragment first so each lane holds four
// consecutive keys of one query row); the row max and sum are butterflies over
// the four lanes that share a row; P = exp(scale * (S - max)) goes to LDS as
// bf16 and O = P V runs on the matrix cores again; O is divided by the row sum
// in fp32 and stored.  Keys past seq are masked to -inf (zero K / V rows),
// queries past seq are computed on zero rows and not stored.
// ---------------------------------------------------------------------------
constexpr int AM_Q = 64, AM_K = 128, AM_D = 64;
constexpr int AM_LD = AM_D + 8;     // bf16 row stride of Q and K (144 bytes)
constexpr int AM_LP = AM_K + 8;     // bf16 row stride of V^T and P (272 bytes)

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t lds8(const __bf16* p) { return *reinterpret_cast<const bf16x8_t*>(p); }

__global__ __launch_bounds__(256) void attention_mfma_kernel(const __bf16* __restrict__ qkv, __bf16* __restrict__ y,
                                                             int seq, int heads, float scale, int n_tiles) {
    // P reuses the Q and K space once S = Q K^T is done (45 KB in all: three blocks per CU)
    static_assert(4 * 16 * AM_LP <= (AM_Q + AM_K) * AM_LD, "P fits where Q and K were");
    __shared__ __attribute__((aligned(16))) __bf16 sqk[(AM_Q + AM_K) * AM_LD];
    __shared__ __attribute__((aligned(16))) __bf16 svt[AM_D * AM_LP];
    __bf16* const sq = sqk;
    __bf16* const sk = sqk + AM_Q * AM_LD;
    __bf16* const sp = sqk;
    // The XCDs take blocks round-robin: number the tiles so that each XCD runs a contiguous
    // range, and the query tiles of one (batch, head) -- which read the same K and V -- run
    // on the same XCD at about the same time, K and V coming from its L2 after the first.
    const int qtiles = (seq + AM_Q - 1) / AM_Q;
    const int tiles = gridDim.x;                       // a multiple of 8 (padded by the launcher)
    const int ti = static_cast<int>(blockIdx.x % 8) * (tiles / 8) + static_cast<int>(blockIdx.x / 8);
    if (ti >= n_tiles) return;
    const int qt = ti % qtiles, bh = ti / qtiles;
    const int b = bh / heads, h = bh % heads;
    const int f = heads * AM_D;
    const int64_t row3 = 3 * static_cast<int64_t>(f);
    const __bf16* base = qkv + static_cast<int64_t>(b) * seq * row3 + h * AM_D;
    const int q0 = qt * AM_Q;
    const uint4 zero4 = make_uint4(0, 0, 0, 0);
    // stage: 8 chunks of 8 dims per row
    for (int i = threadIdx.x; i < AM_Q * 8; i += 256) {
        const int r = i >> 3, c = i & 7, q = q0 + r;
        const uint4 v = q < seq ? *reinterpret_cast<const uint4*>(base + q * row3 + c * 8) : zero4;
        *reinterpret_cast<uint4*>(&sq[r * AM_LD + c * 8]) = v;
    }
    // every key row of the tile is staged (zeros past seq), so the products below run over all
    // AM_K keys with no data-dependent branches; the softmax masks keys >= seq.  A thread takes
    // two adjacent keys, so each V^T word it writes holds both (keys 2p, 2p + 1 of one dim).
    unsigned* svt32 = reinterpret_cast<unsigned*>(svt);
    for (int i = threadIdx.x; i < AM_K / 2 * 8; i += 256) {
        const int kp = i >> 3, c = i & 7, r0 = 2 * kp;
        uint4 k0 = zero4, k1 = zero4, v0 = zero4, v1 = zero4;
        if (r0 < seq) {
            k0 = *reinterpret_cast<const uint4*>(base + r0 * row3 + f + c * 8);
            v0 = *reinterpret_cast<const uint4*>(base + r0 * row3 + 2 * f + c * 8);
        }
        if (r0 + 1 < seq) {
            k1 = *reinterpret_cast<const uint4*>(base + (r0 + 1) * row3 + f + c * 8);
            v1 = *reinterpret_cast<const uint4*>(base + (r0 + 1) * row3 + 2 * f + c * 8);
        }
        *reinterpret_cast<uint4*>(&sk[r0 * AM_LD + c * 8]) = k0;
        *reinterpret_cast<uint4*>(&sk[(r0 + 1) * AM_LD + c * 8]) = k1;
        const unsigned a[4] = {v0.x, v0.y, v0.z, v0.w}, b[4] = {v1.x, v1.y, v1.z, v1.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            svt32[((c * 8 + 2 * e) * AM_LP) / 2 + kp] = (a[e] & 0xffffu) | (b[e] << 16);
            svt32[((c * 8 + 2 * e + 1) * AM_LP) / 2 + kp] = (a[e] >> 16) | (b[e] & 0xffff0000u);
        }
    }
    __syncthreads();

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lr = lane & 15, lg = lane >> 4;          // fragment row, k group
    // S = Q K^T for query rows wave*16 .. +15
    f32x4_t sacc[AM_K / 16];
#pragma unroll
    for (int t = 0; t < AM_K / 16; ++t) sacc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < AM_D / 32; ++ks) {
        const bf16x8_t qa = lds8(&sq[(wave * 16 + lr) * AM_LD + ks * 32 + lg * 8]);
#pragma unroll
        for (int t = 0; t < AM_K / 16; ++t) {
            const bf16x8_t kb = lds8(&sk[(t * 16 + lr) * AM_LD + ks * 32 + lg * 8]);
            sacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb, qa, sacc[t], 0, 0, 0);
        }
    }
    // softmax over the keys of row lr: this lane holds keys 16 t + 4 lg + e
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < AM_K / 16; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int key = t * 16 + lg * 4 + e;
            if (key >= seq) sacc[t][e] = -INFINITY;
            mx = fmaxf(mx, sacc[t][e]);
        }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    __syncthreads();                                   // every wave is done with Q and K: P goes there
    float sum = 0.0f;
    __bf16* prow = &sp[(wave * 16 + lr) * AM_LP];
#pragma unroll
    for (int t = 0; t < AM_K / 16; ++t) {
        float pe[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            pe[e] = sacc[t][e] == -INFINITY ? 0.0f : __expf(scale * (sacc[t][e] - mx));
            sum += pe[e];
        }
        const __bf16 pb[4] = {(__bf16)pe[0], (__bf16)pe[1], (__bf16)pe[2], (__bf16)pe[3]};
        *reinterpret_cast<uint2*>(&prow[t * 16 + lg * 4]) = *reinterpret_cast<const uint2*>(pb);
    }
    sum += __shfl_xor(sum, 16, 64);
    sum += __shfl_xor(sum, 32, 64);
    __syncthreads();                                   // P rows written before their fragment reads
    // O = P V: dims 16 dt + 4 lg + e of row lr
    f32x4_t oacc[AM_D / 16];
#pragma unroll
    for (int dt = 0; dt < AM_D / 16; ++dt) oacc[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < AM_K / 32; ++ks) {
        const bf16x8_t pa = lds8(&sp[(wave * 16 + lr) * AM_LP + ks * 32 + lg * 8]);
#pragma unroll
        for (int dt = 0; dt < AM_D / 16; ++dt) {
            const bf16x8_t vb = lds8(&svt[(dt * 16 + lr) * AM_LP + ks * 32 + lg * 8]);
            oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vb, pa, oacc[dt], 0, 0, 0);
        }
    }
    const int q = q0 + wave * 16 + lr;
    if (q >= seq) return;
    const float inv = 1.0f / sum;
    __bf16* out = y + (static_cast<int64_t>(b) * seq + q) * f + h * AM_D;
#pragma unroll
    for (int dt = 0; dt < AM_D / 16; ++dt) {
        const __bf16 ob[4] = {(__bf16)(oacc[dt][0] * inv), (__bf16)(oacc[dt][1] * inv), (__bf16)(oacc[dt][2] * inv),
                              (__bf16)(oacc[dt][3] * inv)};
        *reinterpret_cast<uint2*>(out + dt * 16 + lg * 4) = *reinterpret_cast<const uint2*>(ob);
    }
}

hipError_t launch_attention(const void* qkv, void* y, int batch, int seq, int heads, float scale, int dtype,
                            hipStream_t s) {
    if (seq < 1 || seq > AM_K) return hipErrorInvalidValue;
    if (dtype == MOPAR_BF16) {
        const int n_tiles = batch * heads * ((seq + AM_Q - 1) / AM_Q);
        launch_kernel(attention_mfma_kernel, dim3((n_tiles + 7) / 8 * 8), dim3(256), 0, s,
                      static_cast<const __bf16*>(qkv), static_cast<__bf16*>(y), seq, heads, scale, n_tiles);
    } else {
        launch_kernel(attention_kernel<float>, dim3(batch * heads), dim3(ATT_MAXS), 0, s,
                      static_cast<const float*>(qkv), static_cast<float*>(y), seq, heads, scale);
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Raw copy (the lossless boundary codec) and zero fill, 16-byte vectors with a
// byte tail.
// ---------------------------------------------------------------------------
__global__ void copy_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t n16) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n16;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
        dst[i] = src[i];
}
__global__ void copy_tail_kernel(const unsigned char* src, unsigned char* dst, int64_t n) {
    const int64_t i = threadIdx.x;
    if (i < n) dst[i] = src[i];
}
__global__ void fill_kernel(uint4* __restrict__ dst, int64_t n16, unsigned v) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n16;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x)
        dst[i] = make_uint4(v, v, v, v);
}
__global__ void fill_tail_kernel(unsigned char* dst, int64_t n, unsigned char v) {
    const int64_t i = threadIdx.x;
    if (i < n) dst[i] = v;
}

static unsigned stream_blocks(int64_t n16) {
    int64_t b = (n16 + 255) / 256;
    if (b > 256 * 16) b = 256 * 16;     // grid-stride beyond 16 blocks per CU
    return static_cast<unsigned>(b < 1 ? 1 : b);
}

hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t s) {
    const int64_t n16 = static_cast<int64_t>(bytes / 16);
    if (n16 > 0)
        launch_kernel(copy_kernel, dim3(stream_blocks(n16)), dim3(256), 0, s, static_cast<const uint4*>(src),
                           static_cast<uint4*>(dst), n16);
    const int64_t tail = static_cast<int64_t>(bytes % 16);
    if (tail)
        launch_kernel(copy_tail_kernel, dim3(1), dim3(16), 0, s,
                           static_cast<const unsigned char*>(src) + n16 * 16,
                           static_cast<unsigned char*>(dst) + n16 * 16, tail);
    return hipGetLastError();
}

hipError_t launch_fill_bytes(void* p, size_t bytes, unsigned char value, hipStream_t s) {
    const int64_t n16 = static_cast<int64_t>(bytes / 16);
    if (n16 > 0)
        launch_kernel(fill_kernel, dim3(stream_blocks(n16)), dim3(256), 0, s, static_cast<uint4*>(p), n16,
                      0x01010101u * value);
    const int64_t tail = static_cast<int64_t>(bytes % 16);
    if (tail)
        launch_kernel(fill_tail_kernel, dim3(1), dim3(16), 0, s, static_cast<unsigned char*>(p) + n16 * 16, tail,
                      value);
    return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s) { return launch_fill_bytes(p, bytes, 0, s); }

// ---------------------------------------------------------------------------
// One autoencoder codec layer whose input width is not a whole number of 16-byte
// chunks (the matrix-core GEMM streams 16-byte chunks of every row, so it needs
// that width on the granule): y[p][o] = b[o] + sum_c w[o][c] x[p][c], one thread
// per (position, output channel), the sum over c in ascending order in float32.
// Such layers are tiny (a few channels per position), so the vector ALUs serve.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void codec_narrow_kernel(const T* __restrict__ x, const T* __restrict__ w,
                                                           const T* __restrict__ b, T* __restrict__ y,
                                                           unsigned total, int cin, int cout) {
    const unsigned i = blockIdx.x * 256u + threadIdx.x;
    if (i >= total) return;
    const unsigned p = i / static_cast<unsigned>(cout);
    const int o = static_cast<int>(i - p * static_cast<unsigned>(cout));
    const T* xr = x + static_cast<int64_t>(p) * cin;
    const T* wr = w + static_cast<int64_t>(o) * cin;
    float acc = b ? to_f(b[o]) : 0.0f;
    for (int c = 0; c < cin; ++c) acc += to_f(wr[c]) * to_f(xr[c]);
    y[i] = from_f<T>(acc);
}

hipError_t launch_codec_narrow(const void* x, const void* w, const void* b, void* y, int64_t positions, int cin,
                               int cout, int dtype, hipStream_t s) {
    const int64_t total = positions * cout;
    if (total <= 0) return hipSuccess;
    if (total >= (int64_t(1) << 31)) return hipErrorInvalidValue;   // 32-bit thread index
    const dim3 grid(blocks_for(total, 256));
    if (dtype == MOPAR_BF16)
        launch_kernel(codec_narrow_kernel<__bf16>, grid, dim3(256), 0, s, static_cast<const __bf16*>(x),
                      static_cast<const __bf16*>(w), static_cast<const __bf16*>(b), static_cast<__bf16*>(y),
                      static_cast<unsigned>(total), cin, cout);
    else
        launch_kernel(codec_narrow_kernel<float>, grid, dim3(256), 0, s, static_cast<const float*>(x),
                      static_cast<const float*>(w), static_cast<const float*>(b), static_cast<float*>(y),
                      static_cast<unsigned>(total), cin, cout);
    return hipGetLastError();
}

size_t dtype_size(int dtype) { return dtype == MOPAR_BF16 ? 2 : 4; }

}  // namespace mopar
