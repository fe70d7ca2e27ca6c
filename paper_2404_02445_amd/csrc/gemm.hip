// MFMA GEMM for gfx950: the resource-dominant operators (conv as implicit GEMM
// over NHWC activations, linear layers), the boundary autoencoder and the
// LSTM recurrence all run through this kernel.
//
//   C[m, n] = epilogue( sum_k A[m, k] * B[n, k] )
//
// A is [M][K]: a dense row-major matrix or the im2col view of an NHWC image
// (k runs over (r, s, c) with c fastest).  B is [N][K] row-major.
//
// Horizontal sub-slicing (the k equal-size sub-slices of an RD operator): a
// block's sub-slice index selects output columns [lo, hi) and weight rows
// [lo, hi), split as mopar_subslice_range does; each sub-slice is tiled on its
// own and masked at hi.  What fixes the arithmetic -- the MFMA shape, the order
// of the 32-wide k steps, the split-K boundaries (in 64-element units) and the
// order partial sums are added -- depends only on (M, N, K) and the dtype, never
// on the tile shape, the stage depth or the sub-slice, so every output element
// goes through the same fp32 operations whatever k is: sub-sliced output equals
// the unsplit output bit for bit.
//
// Data path.  Operands stream from HBM straight into LDS with buffer_load_dwordx4
// ... lds (16 bytes per lane, no VGPR staging), NS stages deep; a stage holds one
// sub-stage (one per wave on the K-split tiles) and costs one barrier.  A
// sub-stage holds 64 bf16 (32 float) of k for
// every row: 128 bytes, one cache line.  Each load instruction fetches 8 whole rows
// (the DMA writes lane l's 16 bytes to slot l of a 1 KB LDS block); lanes take the
// chunks of a row in XOR-swizzled order (chunk (l % 8) ^ row), so the ds_read_b128
// of an MFMA fragment -- 16 rows, one chunk each -- hits distinct banks.  Each
// operand is a raw buffer resource: a lane's offset is fixed at set-up, the k
// advance of dense operands is a scalar offset, and out-of-range chunks (image
// padding, the K tail) use an offset past the resource, which writes zeros without
// a memory access -- every lane issues the same loads, so the wait counts are
// exact.  The waves run v_mfma_f32_16x16x32_bf16 (bf16) or v_mfma_f32_16x16x4_f32
// (fp32) on their wave tile, with the weight fragment as the first operand: each
// lane ends up holding four consecutive output columns of one row.  The
// accumulators start at the bias (loaded before the operand stages); the epilogue
// stages the fp32 tile through LDS so that each thread finishes whole 8-column
// chunks (residual, activation, one 16-byte store), except that tiles of 32
// columns or fewer store straight from the MFMA layout; the LSTM cell works on the
// MFMA layout directly.
//
// Blocks are numbered so that the eight XCDs (which take blocks round-robin)
// each receive a contiguous run of tiles, grouped eight m-tiles at a time so
// that the blocks an XCD runs together share A rows and B rows in its L2.
#include <type_traits>

#include "internal.h"

namespace mopar {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef const __attribute__((address_space(1))) void* gptr_t;

template <typename T> struct Elt;
template <> struct Elt<__bf16> { static constexpr int EPC = 8; };   // elements per 16-byte chunk
template <> struct Elt<float> { static constexpr int EPC = 4; };

// 32 zero bytes: the source of absent epilogue operands.
__device__ __attribute__((aligned(16))) const unsigned int kZeroChunk[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};

// Raw buffer resources: word 3 of the descriptor (32-bit data format) and the lane offset
// that lies past every resource (operand sizes are below 2^31 bytes) and so reads zeros.
constexpr int kRsrcWord3 = 0x00020000;
// m tiles per group in the XCD-local block order
constexpr int kGroupM = 8;
constexpr unsigned kOOB = 0x80000000u;

// Touch every 64-byte line of a kernel's BYTES of arguments at entry: their scalar-cache misses
// then overlap in one wait instead of arriving phase by phase as fields are first used.
template <size_t BYTES>
__device__ __forceinline__ void touch_kernargs() {
    const auto* ka = (const __attribute__((address_space(4))) unsigned*)(__builtin_amdgcn_kernarg_segment_ptr());
    unsigned x = 0;
#pragma unroll
    for (int o = 0; o < static_cast<int>(BYTES / 4); o += 16) x |= ka[o];
    asm volatile("" ::"s"(x));
}

// f(std::integral_constant<int, i>) for i = 0 .. N-1, unrolled at compile time
template <int N, typename F, int I = 0>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<N, F, I + 1>(static_cast<F&&>(f));
    }
}

__device__ __forceinline__ float ld_f(const __bf16* p, int64_t i) {
    unsigned short u = reinterpret_cast<const unsigned short*>(p)[i];
    return __uint_as_float(static_cast<unsigned>(u) << 16);
}
__device__ __forceinline__ float ld_f(const float* p, int64_t i) { return p[i]; }

// whether q is aligned to a whole vector of four elements (8 bytes for bf16, 16 for float)
template <typename T>
__device__ __forceinline__ bool aligned4(const T* q) { return (reinterpret_cast<uintptr_t>(q) & (4 * sizeof(T) - 1)) == 0; }

// four consecutive elements (vector load when the address is aligned)
template <typename T>
__device__ __forceinline__ void ld4(const T* p, int64_t i, int nvalid, float* v) {
    if constexpr (sizeof(T) == 2) {
        if (nvalid == 4 && aligned4(p + i)) {
            const uint2 r = *reinterpret_cast<const uint2*>(p + i);
            v[0] = __uint_as_float(r.x << 16);
            v[1] = __uint_as_float(r.x & 0xffff0000u);
            v[2] = __uint_as_float(r.y << 16);
            v[3] = __uint_as_float(r.y & 0xffff0000u);
            return;
        }
    } else {
        if (nvalid == 4 && aligned4(p + i)) {
            const f32x4 r = *reinterpret_cast<const f32x4*>(p + i);
            v[0] = r[0], v[1] = r[1], v[2] = r[2], v[3] = r[3];
            return;
        }
    }
    for (int q = 0; q < 4; ++q) v[q] = q < nvalid ? ld_f(p, i + q) : 0.0f;
}

__device__ __forceinline__ float sigmoidf_(float v) { return 1.0f / (1.0f + __expf(-v)); }

// erf by formula 7.1.26 of Abramowitz and Stegun's Handbook of Mathematical Functions (absolute
// error at most 1.5e-7): erf(x) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) e^(-x^2) with
// t = 1 / (1 + p x) for x >= 0, odd in x.  Branch-free (the hardware reciprocal and exponential,
// about 1 ulp each, and five multiply-adds), where the library's erf takes several times the
// instructions and branches on |x|: in GELU epilogues it cost a quarter of BERT-base's FFN1
// (9.5 of 39.7 us).  The error is far below the rounding of GELU's result to bf16 and, relative
// to the output's scale, below float32's.
__device__ __forceinline__ float erf_as(float x) {
    const float ax = __builtin_fabsf(x);
    const float t = __builtin_amdgcn_rcpf(1.0f + 0.3275911f * ax);
    const float poly =
        t * (0.254829592f + t * (-0.284496736f + t * (1.421413741f + t * (-1.453152027f + t * 1.061405429f))));
    return __builtin_copysignf(1.0f - poly * __expf(-ax * ax), x);
}

__device__ __forceinline__ float act_f(float v, int act) {
    if (act == MOPAR_ACT_RELU) return v > 0.0f ? v : 0.0f;
    if (act == MOPAR_ACT_GELU) return 0.5f * v * (1.0f + erf_as(v * 0.70710678118654752f));
    return v;
}

// four consecutive elements to c + idx (vector store when the address is aligned: a branch
// written into a concatenated tensor may start at any channel)
template <typename T>
__device__ __forceinline__ void store4(T* c, int64_t idx, const float* v, int nvalid) {
    if constexpr (sizeof(T) == 2) {
        if (nvalid == 4 && aligned4(c + idx)) {
            const bf16x4 o = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
            *reinterpret_cast<bf16x4*>(c + idx) = o;
            return;
        }
    } else {
        if (nvalid == 4 && aligned4(c + idx)) {
            *reinterpret_cast<f32x4*>(c + idx) = f32x4{v[0], v[1], v[2], v[3]};
            return;
        }
    }
    for (int q = 0; q < nvalid; ++q) c[idx + q] = static_cast<T>(v[q]);
}

// eight consecutive elements as raw bits (one 16-byte load for bf16, two for float32)
template <typename T> struct Raw8 { uint4 w[sizeof(T) / 2]; };

__device__ __forceinline__ bool aligned16(const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; }

template <typename T>
__device__ __forceinline__ void unpack8(const Raw8<T>& r, float (&v)[8]) {
    if constexpr (sizeof(T) == 2) {
        const unsigned w[4] = {r.w[0].x, r.w[0].y, r.w[0].z, r.w[0].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            v[2 * q] = __uint_as_float(w[q] << 16);
            v[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
        }
    } else {
        const unsigned w[8] = {r.w[0].x, r.w[0].y, r.w[0].z, r.w[0].w, r.w[1].x, r.w[1].y, r.w[1].z, r.w[1].w};
#pragma unroll
        for (int q = 0; q < 8; ++q) v[q] = __uint_as_float(w[q]);
    }
}

// v[0..7] = p[i..i+7] for the first nvalid elements, 0 after them (and everywhere when p is null)
template <typename T>
__device__ __forceinline__ void load8(const T* p, int64_t i, int nvalid, float (&v)[8]) {
    if (p && nvalid == 8 && aligned16(p + i)) {
        unpack8<T>(*reinterpret_cast<const Raw8<T>*>(p + i), v);
        return;
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = (p && q < nvalid) ? ld_f(p, i + q) : 0.0f;
}

// four consecutive elements as raw bits (8 bytes for bf16, 16 for float)
template <typename T> struct Raw4Sel { using type = uint4; };
template <> struct Raw4Sel<__bf16> { using type = uint2; };
template <typename T> using Raw4 = typename Raw4Sel<T>::type;

// the 4 elements at q (8-byte aligned for bf16, 16 for float), or zeros from the zero page when
// q is null: one unconditional load either way
template <typename T>
__device__ __forceinline__ Raw4<T> load_raw4(const T* q, const void* zero_page) {
    // through a global-address-space pointer, so it is a global (not flat) load
    const void* src = q ? static_cast<const void*>(q) : zero_page;
    Raw4<T> r;
    if constexpr (sizeof(T) == 2) {
        const unsigned long long v = *(const __attribute__((address_space(1))) unsigned long long*)(src);
        r.x = static_cast<unsigned>(v);
        r.y = static_cast<unsigned>(v >> 32);
    } else {
        typedef unsigned w4_t __attribute__((ext_vector_type(4)));
        const w4_t v = *(const __attribute__((address_space(1))) w4_t*)(src);
        r.x = v[0], r.y = v[1], r.z = v[2], r.w = v[3];
    }
    return r;
}
template <typename T>
__device__ __forceinline__ void unpack4(const Raw4<T>& r, float (&v)[4]) {
    if constexpr (sizeof(T) == 2) {
        v[0] = __uint_as_float(r.x << 16);
        v[1] = __uint_as_float(r.x & 0xffff0000u);
        v[2] = __uint_as_float(r.y << 16);
        v[3] = __uint_as_float(r.y & 0xffff0000u);
    } else {
        v[0] = __uint_as_float(r.x), v[1] = __uint_as_float(r.y), v[2] = __uint_as_float(r.z), v[3] = __uint_as_float(r.w);
    }
}
// the 4 floats at q (16-byte aligned), or zeros from the zero page when q is null: one
// unconditional global load either way
__device__ __forceinline__ f32x4 load_f32x4(const float* q, const void* zero_page) {
    const void* src = q ? static_cast<const void*>(q) : zero_page;
    return *(const __attribute__((address_space(1))) f32x4*)(src);
}

// p[i .. i+nvalid-1] (zeros after them, and everywhere when p is null), element by element
template <typename T>
__device__ __forceinline__ void ld4_or_zero(const T* p, int64_t i, int nvalid, float (&v)[4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = (p && q < nvalid) ? ld_f(p, i + q) : 0.0f;
}

// the 16 (bf16) or 32 (float) bytes at q, or zeros from the zero page when q is null: one
// unconditional load either way
template <typename T>
__device__ __forceinline__ Raw8<T> load_raw8(const T* q, const void* zero_page) {
    // through a global-address-space pointer, so it is a global (not flat) load
    typedef unsigned w4_t __attribute__((ext_vector_type(4)));
    const auto* src = (const __attribute__((address_space(1))) w4_t*)(q ? static_cast<const void*>(q) : zero_page);
    Raw8<T> r;
#pragma unroll
    for (int h = 0; h < static_cast<int>(sizeof(T)) / 2; ++h) {
        const w4_t v = src[h];
        r.w[h] = make_uint4(v[0], v[1], v[2], v[3]);
    }
    return r;
}

template <typename T>
__device__ __forceinline__ void store8(T* c, int64_t idx, const float (&v)[8], int nvalid) {
    if (nvalid == 8 && aligned16(c + idx)) {
        if constexpr (sizeof(T) == 2) {
            const bf16x8 o = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3],
                              (__bf16)v[4], (__bf16)v[5], (__bf16)v[6], (__bf16)v[7]};
            *reinterpret_cast<bf16x8*>(c + idx) = o;
        } else {
            *reinterpret_cast<f32x4*>(c + idx) = f32x4{v[0], v[1], v[2], v[3]};
            *reinterpret_cast<f32x4*>(c + idx + 4) = f32x4{v[4], v[5], v[6], v[7]};
        }
        return;
    }
    for (int q = 0; q < nvalid; ++q) c[idx + q] = static_cast<T>(v[q]);
}

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// LDS fragment reads.  They are issued as inline asm so the compiler does not
// treat them as readers of the in-flight LDS DMA (it would otherwise drain every
// outstanding global_load_lds before each read, collapsing the pipeline to one
// stage); completion is awaited explicitly with lds_wait(), and pin() ties each
// value to that wait so no use can be scheduled above it.
__device__ __forceinline__ u32x4 lds_read16(unsigned addr) {
    u32x4 v;
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
    return v;
}
// One 16-byte chunk per lane from the raw buffer [base, base + size) at byte offset voff + soff
// (soff wave-uniform) into LDS slot lane of the 1 KB block at dst; an offset voff >= size
// writes zeros.  (The resource is built here, in a plain device function, and not in the
// kernel templates.)
__device__ __forceinline__ void buffer_load_lds(const void* base, unsigned size, lds_ptr_t dst, unsigned voff,
                                                unsigned soff) {
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                                                      static_cast<int>(size), kRsrcWord3);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, soff, 0, 0);
}

template <int OFF>
__device__ __forceinline__ u32x4 lds_read16_at(unsigned addr) {
    static_assert(OFF >= 0 && OFF < 65536, "ds offset");
    u32x4 v;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(OFF));
    return v;
}
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
template <int N>
__device__ __forceinline__ void lds_wait_until() {
    static_assert(N >= 0 && N <= 15, "lgkmcnt range");
    asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void pin(u32x4& v) { asm volatile("" : "+v"(v)); }

// wait until at most `r` of this wave's stages (L loads each) are still in flight
template <int L>
__device__ __forceinline__ void wait_stages(int r) {
    switch (r) {
        case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
        case 1: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(L) : "memory"); break;
        case 2: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * L) : "memory"); break;
        case 3: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(3 * L) : "memory"); break;
        case 4: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(4 * L < 63 ? 4 * L : 63) : "memory"); break;
        case 5: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(5 * L < 63 ? 5 * L : 63) : "memory"); break;
        case 6: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(6 * L < 63 ? 6 * L : 63) : "memory"); break;
        default: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(7 * L < 63 ? 7 * L : 63) : "memory"); break;
    }
}

// KS > 1: the KS waves of a block share one wave tile (the whole block tile) and split K
// instead: a stage holds KH = KS sub-stages and wave w computes sub-stage w of each, so the
// serial K loop is KS times shorter; the waves' sums are added in wave order at the end.
template <typename T, int BM, int BN, int WM, int WN, int NS, int KH, int KS, bool CONV>
__global__ __launch_bounds__(WM * WN * KS * 64) void gemm_kernel(const GemmParams p) {
    constexpr int EPC = Elt<T>::EPC;
    constexpr int BK = 8 * EPC;                 // K elements per sub-stage: two 32-wide (bf16) k steps
    constexpr int TM = BM / WM, TN = BN / WN;   // wave tile
    constexpr int FM = TM / 16, FN = TN / 16;   // 16x16 MFMA tiles per wave
    constexpr int NBA = BM / 16 * 2, NBB = BN / 16 * 2;
    constexpr int NBLK = NBA + NBB;             // 1 KB fragment blocks per stage
    constexpr int NW = WM * WN * KS, NT = NW * 64;   // waves and threads per block
    constexpr int LA = (NBA + NW - 1) / NW, LB = (NBB + NW - 1) / NW;   // load slots per wave
    constexpr int LMIN = NBA / NW + NBB / NW;   // loads per sub-stage issued by every wave
    constexpr int STAGE = NBLK * 64;            // uint4 per sub-stage
    constexpr int SSTAGE = KH * STAGE;          // uint4 per stage: KH sub-stages, one barrier
    static_assert((NW == 4 || NW == 8) && FM >= 1 && FN >= 1 && NS >= 2 && NS <= 9 && LMIN >= 1, "tile");
    static_assert(KH == 1 || KH == 2 || KH == 4, "sub-stages per stage");
    static_assert(KS == KH && (KS == 1 || (WM == 1 && WN == 1)), "K split across waves: one sub-stage per wave");
    static_assert((NS - 2) * LMIN * KH <= 63, "vmcnt range");

    constexpr int LDT = BN + 4;                 // fp32 row stride of the staged output tile (padded)
    constexpr int TILE_U4 = (KS * BM * LDT + 3) / 4;   // staged output tile(s), one per K-split wave
    constexpr int LDS_U4 = NS * SSTAGE > TILE_U4 ? NS * SSTAGE : TILE_U4;
    __shared__ uint4 lds[LDS_U4];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // scalar: load blocks are wave-uniform
    const int wt = KS > 1 ? 0 : wave;           // wave-tile index
    const int kw = KS > 1 ? wave : 0;           // K-split index
    const int wm = wt / WN, wn = wt % WN;

    // --- block -> (m tile, split, sub-slice, n tile), XCD-grouped -------------------------
    // (all divisions by launch constants go through precomputed multipliers)
    touch_kernargs<sizeof(GemmParams)>();
    const unsigned t = (blockIdx.x % 8) * static_cast<unsigned>(p.g_per_xcd) + blockIdx.x / 8;
    if (t >= static_cast<unsigned>(p.g_total)) return;
    // within an XCD's run, tiles go in groups of GM m-tiles x every column (split, sub-slice,
    // n-tile), m fastest: the blocks resident together share both A rows and B rows in L2
    constexpr int GM = kGroupM;
    const unsigned group = p.g_div_group.div(t);
    const unsigned within = t - group * static_cast<unsigned>(GM * p.g_cols);
    const bool last = static_cast<int>(group) == (p.g_mt - 1) / GM;   // the last group may be short
    const unsigned gm = last ? static_cast<unsigned>(p.g_mt - group * GM) : GM;
    const unsigned colu = last ? p.g_div_last.div(within) : within / GM;
    const int mti = static_cast<int>(group * GM + (within - colu * gm));
    const unsigned c1 = p.g_div_nt.div(colu);
    const int nti = static_cast<int>(colu - c1 * static_cast<unsigned>(p.g_nt));
    const unsigned c2 = p.g_div_ksub.div(c1);
    const int j = static_cast<int>(c1 - c2 * static_cast<unsigned>(p.ksub));
    const int split = static_cast<int>(c2);

    const int q = p.g_q, rr = p.g_rr;
    const int n_lo = j * q + min(j, rr), n_hi = (j + 1) * q + min(j + 1, rr);
    const int n0 = n_lo + nti * BN;
    if (n0 >= n_hi) return;                     // block-uniform, before any barrier
    // rows fit in 32 bits (M <= 2^31 - 256, checked at launch); output offsets are 64-bit
    const int Mi = static_cast<int>(p.M);
    const int m0 = mti * BM;

    // this split's sub-stages [u0, u1): boundaries in BK units, whatever KH is
    const int nk = p.g_nk;
    const int u0 = static_cast<int>(p.g_div_splits.div(static_cast<unsigned>(nk * split)));
    const int u1 = static_cast<int>(p.g_div_splits.div(static_cast<unsigned>(nk * (split + 1))));
    const int nst = (u1 - u0 + KH - 1) / KH;    // stages; sub-stages past u1 re-read u0, run no MFMA

    // --- operand loads ----------------------------------------------------------------------
    // Each operand is read through a raw buffer resource: a lane's chunk address is a fixed
    // per-lane byte offset (VGPR) plus a per-sub-stage offset that only the scalar unit
    // advances (dense operands), and a lane whose offset is kOOB -- past the resource's size
    // -- writes zeros to LDS without touching memory (image padding, K tail).
    // Load block blk of a sub-stage covers 8 rows x 128 bytes (whole cache lines): lane l
    // loads row 8 * blk + l / 8, k chunk cl = (l % 8) ^ (l / 8) -- the XOR swizzle that keeps
    // the fragment reads conflict-free -- into LDS slot l of the block.  Wave w loads A blocks
    // w, w + NW, ... and B blocks w, w + NW, ...: slots are fixed at compile time, and only a
    // last, partial round of slots tests the wave index.
    const int cl = (lane & 7) ^ (lane >> 3);    // this lane's chunk of every sub-stage, 0..7
    // Rows past M (A) or past the sub-slice (B) load a real row (the last valid one) instead:
    // the products they feed are never stored.
    // Dense A and B: voff = byte offset of (row, chunk cl of sub-stage 0).  Conv A: voff =
    // offset of the window's top-left pixel (two's complement when the window starts in the
    // padding), with the window corner (hb, wb) for the bounds test.
    unsigned voffA[LA], voffB[LB];
    int hb[LA], wb[LA];
#pragma unroll
    for (int i = 0; i < LA; ++i) {
        const int blk = min(wave + NW * i, NBA - 1);
        const int m = m0 + blk * 8 + (lane >> 3);
        const int mc = m < Mi ? m : Mi - 1;
        hb[i] = wb[i] = 0;
        if constexpr (CONV) {
            // M < 2^31, so the pixel decode runs in 32 bits with precomputed divisors
            const unsigned mu = static_cast<unsigned>(mc);
            const unsigned img = p.div_hw.div(mu);
            const unsigned rem = mu - img * static_cast<unsigned>(p.out_h * p.out_w);
            const unsigned ho = p.div_w.div(rem), wo = rem - ho * static_cast<unsigned>(p.out_w);
            hb[i] = static_cast<int>(ho) * p.stride - p.pad;
            wb[i] = static_cast<int>(wo) * p.stride - p.pad;
            const int pix = (static_cast<int>(img) * p.img_h + hb[i]) * p.img_w + wb[i];
            voffA[i] = static_cast<unsigned>(pix) * static_cast<unsigned>(p.cs * sizeof(T));
        } else {
            // (A spans less than 2^31 bytes, so the offset of row mc fits in 32 bits)
            voffA[i] = static_cast<unsigned>(mc) * static_cast<unsigned>(p.lda * sizeof(T)) + static_cast<unsigned>(cl * 16);
        }
    }
#pragma unroll
    for (int i = 0; i < LB; ++i) {
        const int blk = min(wave + NW * i, NBB - 1);
        const int n = n0 + blk * 8 + (lane >> 3);
        const int nc = n < n_hi ? n : n_hi - 1;
        voffB[i] = static_cast<unsigned>(nc) * static_cast<unsigned>(p.K * sizeof(T)) + static_cast<unsigned>(cl * 16);
    }

    // im2col coordinates (tap row, tap column, channel) of this lane's chunk, advanced
    // incrementally by one sub-stage: BK = (dqr * kw + dqc) * cs + dc elements
    int tr = 0, tcol = 0, tci = 0;
    const int dqr = p.dqr, dqc = p.dqc, dc = p.dc;
    if (CONV) {
        const unsigned k = static_cast<unsigned>(u0 * BK + cl * EPC);
        const unsigned tap = p.div_cs.div(k);
        tci = static_cast<int>(k - tap * static_cast<unsigned>(p.cs));
        const unsigned r = p.div_kw.div(tap);
        tr = static_cast<int>(r);
        tcol = static_cast<int>(tap - r * static_cast<unsigned>(p.kw));
    }
    auto advance = [&]() {
        tci += dc;
        const int carry = tci >= p.cs ? 1 : 0;
        tci -= carry * p.cs;
        tcol += dqc + carry;                    // < 2 kw: one wrap at most
        tr += dqr;
        if (tcol >= p.kw) {
            tcol -= p.kw;
            ++tr;
        }
    };

    // Loads of sub-stage kt (conv coordinates must be those of kt) into LDS at dst.  A dead
    // sub-stage (past the split: its MFMAs are skipped) re-reads sub-stage u0, so that every
    // sub-stage issues the same loads and the wait counts stay exact.
    const int ktail = (p.K % BK) ? nk - 1 : nk;   // the one sub-stage whose chunks may pass K
    auto issue = [&](int kt, uint4* dst, bool live) {
        const int ku = live ? kt : u0;
        const unsigned soff = static_cast<unsigned>(ku) * (BK * sizeof(T));
        const bool tail = ku == ktail;          // uniform
        const bool kin = !tail || ku * BK + cl * EPC < p.K;
        const unsigned koff = CONV ? static_cast<unsigned>(((tr * p.img_w + tcol) * p.cs + tci) * sizeof(T)) : 0u;
#pragma unroll
        for (int i = 0; i < LA; ++i) {
            if (NBA % NW != 0 && i == LA - 1 && wave + NW * i >= NBA) break;   // wave-uniform
            unsigned v;
            if constexpr (CONV) {
                const bool ok = kin && static_cast<unsigned>(hb[i] + tr) < static_cast<unsigned>(p.img_h) &&
                                static_cast<unsigned>(wb[i] + tcol) < static_cast<unsigned>(p.img_w);
                v = ok ? voffA[i] + koff : kOOB;
            } else {
                v = kin ? voffA[i] : kOOB;
            }
            buffer_load_lds(p.A, p.a_bytes, (lds_ptr_t)(dst + (wave + NW * i) * 64), v, CONV ? 0u : soff);
        }
#pragma unroll
        for (int i = 0; i < LB; ++i) {
            if (NBB % NW != 0 && i == LB - 1 && wave + NW * i >= NBB) break;
            buffer_load_lds(p.B, p.b_bytes, (lds_ptr_t)(dst + (NBA + wave + NW * i) * 64), kin ? voffB[i] : kOOB, soff);
        }
    };
    // stage st: sub-stages u0 + st * KH + h into buffer buf, conv coordinates advanced past them
    auto issue_stage = [&](int st, int buf) {
#pragma unroll
        for (int h = 0; h < KH; ++h) {
            const int kt = u0 + st * KH + h;
            issue(kt, &lds[buf * SSTAGE + h * STAGE], kt < u1);
            if (CONV) advance();
        }
    };

    f32x4 acc[FM][FN];
#pragma unroll
    for (int a = 0; a < FM; ++a)
#pragma unroll
        for (int b = 0; b < FN; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

    // --- epilogue set-up ---------------------------------------------------------------------
    // MFMA layout: lane holds row mrow[a], columns ncol[b]..+3
    int mrow[FM];
    int ncol[FN], nval[FN];
#pragma unroll
    for (int a = 0; a < FM; ++a) mrow[a] = m0 + wm * TM + a * 16 + (lane & 15);
#pragma unroll
    for (int b = 0; b < FN; ++b) {
        ncol[b] = n0 + wn * TN + b * 16 + (lane >> 4) * 4;
        nval[b] = max(0, min(4, n_hi - ncol[b]));
    }
    // chunk layout (everything else): thread owns 8 consecutive columns c0..c0+7 of tile
    // rows cr, cr + RPP, ...; after the staging through LDS each chunk is one 16-byte store
    constexpr int CPR = BN / 8, RPP = NT / CPR, NCH = (BM + RPP - 1) / RPP;
    const int cc = threadIdx.x % CPR, cr = threadIdx.x / CPR;
    const int c0 = n0 + cc * 8;
    const int cval = max(0, min(8, n_hi - c0));
    const bool direct = p.splits == 1 && p.epi == EPI_STD;   // this block finishes its outputs
    // A direct launch starts its accumulators at bias + second bias.  Their raw bits (MFMA
    // layout: 4 columns per lane and fragment) are loaded here, before the operand stages, and
    // added after the prologue: the latency hides under the first stage's.  Each is one load
    // per lane, from the zero page when absent; partial column groups are read element by
    // element up front.  With K split across waves only wave 0 starts from them.  (The residual is added in the epilogue, in
    // the chunk layout whose 16-byte loads cover whole lines: in the MFMA layout its 8-byte
    // loads were measured slower.)
    const T* biasp = static_cast<const T*>(p.bias);
    const T* bias2p = static_cast<const T*>(p.bias2);
    const T* resp = static_cast<const T*>(p.res);
    const bool init_here = direct && (KS == 1 || kw == 0);
    // (Loads whose results a path never reads would leave their registers pending there, and
    // the compiler would then drain every load in flight, operand stages included, when it
    // reuses those registers inside the K loop: each of these loads is issued only under the
    // wave-uniform condition under which it is added.)
    Raw4<T> rb[FN], rb2[FN];
    bool bfast[FN];
    float bslow[FN][4];                         // partial groups: summed bias, read up front
#pragma unroll
    for (int b = 0; b < FN; ++b) {
        bfast[b] = nval[b] == 4;
        if (init_here) {
            rb[b] = load_raw4<T>(bfast[b] && biasp ? biasp + ncol[b] : nullptr, kZeroChunk);
            rb2[b] = load_raw4<T>(bfast[b] && bias2p ? bias2p + ncol[b] : nullptr, kZeroChunk);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) bslow[b][e] = 0.0f;
        // (element loads under a per-lane branch: done before any operand load is in flight,
        // since the wait they need would otherwise drain the operand stages too)
        if (init_here && !bfast[b]) {
            float bv[4], b2v[4];
            ld4_or_zero<T>(biasp, ncol[b], nval[b], bv);
            ld4_or_zero<T>(bias2p, ncol[b], nval[b], b2v);
#pragma unroll
            for (int e = 0; e < 4; ++e) bslow[b][e] = bv[e] + b2v[e];
        }
    }
    // An LSTM step starts wave 0's accumulators at the gate pre-activations gx (fp32, loaded
    // here in the same way): the epilogue then only applies the cell.
    const bool lstm_here = p.epi == EPI_LSTM && (KS == 1 || kw == 0);
    f32x4 rgx[FM][FN];
    if (lstm_here) {
#pragma unroll
        for (int a = 0; a < FM; ++a)
#pragma unroll
            for (int b = 0; b < FN; ++b) {
                const bool ok = mrow[a] < Mi && nval[b] == 4;
                rgx[a][b] = load_f32x4(ok ? p.gx + static_cast<int64_t>(mrow[a]) * p.ldgx + ncol[b] : nullptr, kZeroChunk);
            }
    }

    // prologue: NS-1 stages in flight (coordinates then stand at stage NS - 1); stages past
    // the split re-read its first sub-stage, and are issued anyway so that the loads in flight
    // at this point do not depend on the path
#pragma unroll
    for (int s = 0; s < NS - 1; ++s) issue_stage(s, s);

    if (lstm_here) {
#pragma unroll
        for (int a = 0; a < FM; ++a)
#pragma unroll
            for (int b = 0; b < FN; ++b) acc[a][b] = rgx[a][b];
    }
    if (init_here) {
#pragma unroll
        for (int b = 0; b < FN; ++b) {
            float bv[4], b2v[4];
            unpack4<T>(rb[b], bv);
            unpack4<T>(rb2[b], b2v);
#pragma unroll
            for (int a = 0; a < FM; ++a)
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[a][b][e] = bfast[b] ? bv[e] + b2v[e] : bslow[b][e];
        }
    }
    // The accumulators now hold values computed from loads; pinning them here makes the
    // compiler settle those loads once, before the K loop.  (Otherwise it treats the
    // accumulators as possibly pending loads inside the loop and waits there for every load
    // in flight, the operand stages just issued included.)
#pragma unroll
    for (int a = 0; a < FM; ++a)
#pragma unroll
        for (int b = 0; b < FN; ++b) asm volatile("" : "+v"(acc[a][b]));

    // LDS byte addresses of this lane's MFMA fragments (row l % 16 of a 16-row block, chunk
    // 4 * ks + l / 16) in stage buffer 0, sub-stage 0, for the wave's first A and B rows;
    // the other fragments sit at compile-time offsets from them
    const unsigned lds0 = static_cast<unsigned>(reinterpret_cast<size_t>((lds_ptr_t)(&lds[0])));
    unsigned fa[2], fb[2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        const unsigned f = lds0 + ((((lane >> 3) & 1) * 64 + (lane & 7) * 8 + ((ks * 4 + (lane >> 4)) ^ (lane & 7))) * 16);
        fa[ks] = f + ((wm * TM) >> 3) * 1024;
        fb[ks] = f + (NBA + ((wn * TN) >> 3)) * 1024;
    }
    auto read_frags = [&](unsigned sbase, int ks, u32x4 (&af)[FM], u32x4 (&bf)[FN]) {
        const unsigned ab = sbase + fa[ks], bb = sbase + fb[ks];
        static_for<FM>([&](auto a) { af[a] = lds_read16_at<a * 2048>(ab); });
        static_for<FN>([&](auto b) { bf[b] = lds_read16_at<b * 2048>(bb); });
    };
    auto mfmas = [&](u32x4 (&af)[FM], u32x4 (&bf)[FN]) {
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
    };

    for (int st = 0; st < nst; ++st) {
        const int buf = st % NS;
        const int later = min(NS - 2, nst - 1 - st);   // stages issued after this one
        wait_stages<LMIN * KH>(later);                 // this wave's share of stage st has landed
        __builtin_amdgcn_s_barrier();                  // every wave's share has; stage st-1 fully consumed
        if (st + NS - 1 < nst) issue_stage(st + NS - 1, (st + NS - 1) % NS);
        const unsigned sbase = buf * SSTAGE * 16;
        u32x4 a0[FM], b0[FN], a1[FM], b1[FN];
        if constexpr (KS > 1) {
            // this wave's sub-stage of the stage (uniform skip when it lies past the split)
            if (u0 + st * KH + kw >= u1) continue;
            const unsigned hb = sbase + kw * STAGE * 16;
            read_frags(hb, 0, a0, b0);
            lds_wait();
#pragma unroll
            for (int a = 0; a < FM; ++a) pin(a0[a]);
#pragma unroll
            for (int b = 0; b < FN; ++b) pin(b0[b]);
            read_frags(hb, 1, a1, b1);
            mfmas(a0, b0);
        } else if constexpr (FM + FN <= 3) {
            // thin wave tiles: both k steps' fragment reads go out together; LDS reads complete
            // in order, so once at most FM + FN are outstanding the first step's have landed
            read_frags(sbase, 0, a0, b0);
            read_frags(sbase, 1, a1, b1);
            lds_wait_until<FM + FN>();
#pragma unroll
            for (int a = 0; a < FM; ++a) pin(a0[a]);
#pragma unroll
            for (int b = 0; b < FN; ++b) pin(b0[b]);
            mfmas(a0, b0);
            __builtin_amdgcn_sched_barrier(0);         // keep these MFMAs ahead of the next wait
        } else {
            // wide wave tiles: holding both steps' fragments would cost the registers that
            // keep two blocks per CU resident; the second step's reads follow the first's wait
            read_frags(sbase, 0, a0, b0);
            lds_wait();
#pragma unroll
            for (int a = 0; a < FM; ++a) pin(a0[a]);
#pragma unroll
            for (int b = 0; b < FN; ++b) pin(b0[b]);
            read_frags(sbase, 1, a1, b1);
            mfmas(a0, b0);
        }
        lds_wait();
#pragma unroll
        for (int a = 0; a < FM; ++a) pin(a1[a]);
#pragma unroll
        for (int b = 0; b < FN; ++b) pin(b1[b]);
        mfmas(a1, b1);
    }

    // --- epilogue --------------------------------------------------------------------------
    // The fp32 tile goes through LDS (row-major, padded rows; one copy per K-split wave,
    // added in wave order when read back).
    float* tile = reinterpret_cast<float*>(lds);
    auto stage_tile = [&]() {
        __syncthreads();                      // every wave is done with the operand stages
#pragma unroll
        for (int a = 0; a < FM; ++a)
#pragma unroll
            for (int b = 0; b < FN; ++b) {
                const int row = wm * TM + a * 16 + (lane & 15), col = wn * TN + b * 16 + (lane >> 4) * 4;
                *reinterpret_cast<f32x4*>(tile + (kw * BM + row) * LDT + col) = acc[a][b];
            }
        __syncthreads();
    };
    auto tile4 = [&](int row, int col) {
        f32x4 v = *reinterpret_cast<const f32x4*>(tile + row * LDT + col);
#pragma unroll
        for (int w = 1; w < KS; ++w) v += *reinterpret_cast<const f32x4*>(tile + (w * BM + row) * LDT + col);
        return v;
    };
    if constexpr (KS > 1) {
        stage_tile();
        // the summed tile back in the MFMA layout, for the row tiles this wave finishes
#pragma unroll
        for (int a = 0; a < FM; ++a)
#pragma unroll
            for (int b = 0; b < FN; ++b)
                if (a % KS == kw) acc[a][b] = tile4(a * 16 + (lane & 15), b * 16 + (lane >> 4) * 4);
    }
    if (p.epi == EPI_LSTM) {
        // gates i, f, g, o of unit n / 4 (n is a multiple of 4 and the whole group is valid),
        // gx already in the sums; with K split across waves, wave w finishes row tiles
        // a = w (mod KS)
        float cprev[FM][FN];
#pragma unroll
        for (int a = 0; a < FM; ++a)
#pragma unroll
            for (int b = 0; b < FN; ++b) {
                const bool ok = a % KS == kw && mrow[a] < Mi && nval[b] == 4;
                const int64_t mm = ok ? mrow[a] : 0;
                const int nn = ok ? ncol[b] : 0;
                cprev[a][b] = p.cstate[mm * (p.N >> 2) + (nn >> 2)];
            }
#pragma unroll
        for (int a = 0; a < FM; ++a)
#pragma unroll
            for (int b = 0; b < FN; ++b) {
                if (a % KS != kw || mrow[a] >= Mi || nval[b] != 4) continue;
                const f32x4 v = acc[a][b];
                const float c = sigmoidf_(v[1]) * cprev[a][b] + sigmoidf_(v[0]) * tanhf(v[2]);
                const int u = ncol[b] >> 2;
                p.cstate[static_cast<int64_t>(mrow[a]) * (p.N >> 2) + u] = c;
                static_cast<T*>(p.C)[static_cast<int64_t>(mrow[a]) * p.ldc + u] = static_cast<T>(sigmoidf_(v[3]) * tanhf(c));
            }
        return;
    }

    // Narrow tiles (32 columns or fewer) store straight from the MFMA layout: a lane's four
    // consecutive columns are one 8-byte (bf16) store, and the LDS round trip costs more than
    // the shorter stores save (measured).
    if constexpr (KS == 1 && BN <= 32) {
        if (direct) {
#pragma unroll
            for (int a = 0; a < FM; ++a)
#pragma unroll
                for (int b = 0; b < FN; ++b) {
                    if (mrow[a] >= Mi || nval[b] == 0) continue;
                    const int64_t idx = static_cast<int64_t>(mrow[a]) * p.ldc + ncol[b];
                    float v[4], rv[4] = {0.f, 0.f, 0.f, 0.f};
                    if (resp) ld4<T>(resp, idx, nval[b], rv);
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = act_f(acc[a][b][e] + rv[e], p.act);
                    if (p.out_f32)
                        store4<float>(static_cast<float*>(p.C), idx, v, nval[b]);
                    else
                        store4<T>(static_cast<T*>(p.C), idx, v, nval[b]);
                }
            return;
        }
    }
    // Otherwise every thread owns whole 8-column chunks of the staged tile: full-line stores.
    if constexpr (KS == 1) stage_tile();
    auto tile8 = [&](int r, float (&v)[8]) {
        const f32x4 lo = tile4(r, cc * 8), hi = tile4(r, cc * 8 + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = lo[e], v[4 + e] = hi[e];
    };
    if (direct) {
        // bias is already in the sums: residual, activation, store.  The residual chunks of
        // all this thread's rows go out together before any is used (a load under each row's
        // own conditions would wait for the one before it); partial or unaligned chunks are
        // read element by element when used.
        Raw8<T> rraw[NCH];
        bool rfast[NCH];
        if (resp) {
#pragma unroll
            for (int i = 0; i < NCH; ++i) {
                const int r = cr + i * RPP;
                const int m = m0 + r;
                const int64_t idx = static_cast<int64_t>(m) * p.ldc + c0;
                rfast[i] = r < BM && m < Mi && cval == 8 && aligned16(resp + idx);
                rraw[i] = load_raw8<T>(rfast[i] ? resp + idx : nullptr, kZeroChunk);
            }
        }
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int r = cr + i * RPP;
            const int m = m0 + r;
            if (r >= BM || m >= Mi || cval == 0) continue;
            float v[8], rsd[8];
            tile8(r, v);
            const int64_t idx = static_cast<int64_t>(m) * p.ldc + c0;
            if (resp && rfast[i])
                unpack8<T>(rraw[i], rsd);
            else
                load8<T>(resp, idx, resp ? cval : 0, rsd);
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = act_f(v[e] + rsd[e], p.act);
            if (p.out_f32)
                store8<float>(static_cast<float*>(p.C), idx, v, cval);
            else
                store8<T>(static_cast<T*>(p.C), idx, v, cval);
        }
        return;
    }

    // split-K: this block's partial sums; splitk_reduce_kernel adds them up in split order
    float* part = p.partial + static_cast<int64_t>(split) * p.M * p.N;
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
        const int r = cr + i * RPP;
        const int m = m0 + r;
        if (r >= BM || m >= Mi || cval == 0) continue;
        float v[8];
        tile8(r, v);
        store8<float>(part, static_cast<int64_t>(m) * p.N + c0, v, cval);
    }
}

// Wide products (bf16, dense A, large M, N and K; see gemm_wide_class): 256 x 256 block tiles on
// v_mfma_f32_32x32x16_bf16.  Four waves each own a 128 x 128 quadrant -- 16 accumulator tiles of
// 32 x 32, 256 registers per lane, which the compiler keeps in the accumulation half of the
// register file -- so one block fills a CU, one wave per SIMD.  (A single wave per SIMD issues
// the 32 x 32 x 16 MFMA at ~90 % of the peak rate but the 16 x 16 x 32 one at ~55 %, measured.)
// A stage holds 64 k (64 KB: 256 rows of A and of B, one cache line each) and costs one
// barrier; two stages in LDS.  Per stage a CU moves 64 KB for 8.4 MFLOP (128 FLOP/B, twice the
// 128 x 128 tile's) and a wave reads 32 KB of fragments for 64 MFMAs.  Each 16-wide k step's
// MFMAs run while the next step's fragments are read, so LDS reads always overlap MFMAs, and the
// next stage's loads are spread over the first k step.  Operand loads (whole-line rows into
// XOR-swizzled LDS blocks) are gemm_kernel's; the MFMA shape is not, so an operator whose
// (M, N, K) puts it here runs here for every sub-slice launch, and every output element sees the
// same operations in the same order whatever the sub-slice count.
constexpr int kWideRowB = 256 * 2 + 16, kWideRowF = 256 * 4 + 16;   // staged output row strides, bytes
constexpr int kWideBStages = 2;                                      // B stages in LDS
constexpr int kWideGroupM = 8;                                       // m tiles per group in the block order
// An accumulator read out where it is used (left to itself the compiler copies many accumulator
// tiles to ordinary registers at once, and spills them)
__device__ __forceinline__ float acc_read(float a) {
    float v;
    asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v) : "a"(a));
    return v;
}
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
template <int NB>
__global__ __launch_bounds__(256, 1) void gemm_wide_kernel(const GemmParams p) {
    using T = __bf16;
    constexpr int BM = 256, BN = 256, TM = 128, TN = 128;
    constexpr int FM = TM / 32, FN = TN / 32;   // 32 x 32 MFMA tiles per wave
    constexpr int NBA = BM / 8, NBB = BN / 8;   // 1 KB blocks (8 rows x 128 bytes) per operand stage
    constexpr int NW = 4;
    constexpr int LA = NBA / NW, LB = NBB / NW; // load slots per wave (8 + 8)
    constexpr int SA = NBA * 64, SB = NBB * 64; // uint4 per A stage and per B stage (32 KB each)
    constexpr int BK = 64;
    static_assert(NB == 2 || NB == 3, "B stages in LDS");
    // LDS: two A stages, then NB B stages; the epilogue's staged tile (256 rows of bf16 or 128 rows
    // of float32, rows padded by 16 bytes) reuses the space
    constexpr int OPS_U4 = 2 * SA + NB * SB;
    constexpr int TILE_U4 = (BM * kWideRowB > TM * kWideRowF ? BM * kWideRowB : TM * kWideRowF) / 16;
    __shared__ uint4 lds[OPS_U4 > TILE_U4 ? OPS_U4 : TILE_U4];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave >> 1, wn = wave & 1;

    touch_kernargs<sizeof(GemmParams)>();
    const unsigned t = (blockIdx.x % 8) * static_cast<unsigned>(p.g_per_xcd) + blockIdx.x / 8;
    if (t >= static_cast<unsigned>(p.g_total)) return;
    constexpr int GM = kWideGroupM;
    const unsigned group = p.g_div_group.div(t);
    const unsigned within = t - group * static_cast<unsigned>(GM * p.g_cols);
    const bool last = static_cast<int>(group) == (p.g_mt - 1) / GM;
    const unsigned gm = last ? static_cast<unsigned>(p.g_mt - group * GM) : GM;
    const unsigned colu = last ? p.g_div_last.div(within) : within / GM;
    const int mti = static_cast<int>(group * GM + (within - colu * gm));
    const unsigned c1 = p.g_div_nt.div(colu);
    const int nti = static_cast<int>(colu - c1 * static_cast<unsigned>(p.g_nt));
    const int j = static_cast<int>(c1);         // one split: the column index is the sub-slice

    const int q = p.g_q, rr = p.g_rr;
    const int n_lo = j * q + min(j, rr), n_hi = (j + 1) * q + min(j + 1, rr);
    const int n0 = n_lo + nti * BN;
    if (n0 >= n_hi) return;
    const int Mi = static_cast<int>(p.M);
    const int m0 = mti * BM;
    const int nk = p.g_nk;                      // >= 1 (K >= 64 here)

    // operand loads: gemm_kernel's layout (8 whole rows per 1 KB block, chunk (l % 8) ^ row)
    const int cl = (lane & 7) ^ (lane >> 3);
    unsigned voffA[LA], voffB[LB];
#pragma unroll
    for (int i = 0; i < LA; ++i) {
        const int m = m0 + (wave + NW * i) * 8 + (lane >> 3);
        const int mc = m < Mi ? m : Mi - 1;
        voffA[i] = static_cast<unsigned>(mc) * static_cast<unsigned>(p.lda * sizeof(T)) + static_cast<unsigned>(cl * 16);
    }
#pragma unroll
    for (int i = 0; i < LB; ++i) {
        const int n = n0 + (wave + NW * i) * 8 + (lane >> 3);
        const int nc = n < n_hi ? n : n_hi - 1;
        voffB[i] = static_cast<unsigned>(nc) * static_cast<unsigned>(p.K * sizeof(T)) + static_cast<unsigned>(cl * 16);
    }
    const int ktail = (p.K % BK) ? nk - 1 : nk;
    uint4* const ldsA = &lds[0];
    uint4* const ldsB = &lds[2 * SA];
    // Load slots 2 i, 2 i + 1 of operand X's stage kt into LDS stage buffer buf.  A stage past
    // the last one re-reads the last one (into a buffer nobody reads), so that every iteration
    // issues the same loads and the wait counts stay exact.
    auto issue_a = [&](int kt, int buf, int i) __attribute__((always_inline)) {
        kt = kt < nk ? kt : nk - 1;
        const unsigned soff = static_cast<unsigned>(kt) * (BK * sizeof(T));
        const bool kin = kt != ktail || kt * BK + cl * 8 < p.K;
#pragma unroll
        for (int s2 = 2 * i; s2 < 2 * i + 2; ++s2)
            buffer_load_lds(p.A, p.a_bytes, (lds_ptr_t)(ldsA + buf * SA + (wave + NW * s2) * 64), kin ? voffA[s2] : kOOB, soff);
    };
    auto issue_b = [&](int kt, int buf, int i) __attribute__((always_inline)) {
        kt = kt < nk ? kt : nk - 1;
        const unsigned soff = static_cast<unsigned>(kt) * (BK * sizeof(T));
        const bool kin = kt != ktail || kt * BK + cl * 8 < p.K;
#pragma unroll
        for (int s2 = 2 * i; s2 < 2 * i + 2; ++s2)
            buffer_load_lds(p.B, p.b_bytes, (lds_ptr_t)(ldsB + buf * SB + (wave + NW * s2) * 64), kin ? voffB[s2] : kOOB, soff);
    };
    static_assert(LA == LB && LA == 2 * FM, "two load slots per row of fragments");

    // MFMA layout (weight fragment first): accumulator register r of tile (a, b) holds output
    // row m = m0 + wm TM + 32 a + l % 32 and column n = n0 + wn TN + 32 b + 8 (r / 4) + 4 (l / 32)
    // + r % 4: four groups of four consecutive columns per lane
    const int lrow = lane & 31, lhalf = lane >> 5;
    // bias + second bias, as gemm_kernel starts a direct launch (partial groups read up front)
    const T* biasp = static_cast<const T*>(p.bias);
    const T* bias2p = static_cast<const T*>(p.bias2);
    Raw4<T> rb[FN][4], rb2[FN][4];
    float bslow[FN][4][4];
#pragma unroll
    for (int b = 0; b < FN; ++b)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int n = n0 + wn * TN + b * 32 + g * 8 + lhalf * 4;
            const int nv = max(0, min(4, n_hi - n));
            const bool fast = nv == 4;
            rb[b][g] = load_raw4<T>(fast && biasp ? biasp + n : nullptr, kZeroChunk);
            rb2[b][g] = load_raw4<T>(fast && bias2p ? bias2p + n : nullptr, kZeroChunk);
            float bv[4], b2v[4];
            ld4_or_zero<T>(biasp, n, fast ? 0 : nv, bv);
            ld4_or_zero<T>(bias2p, n, fast ? 0 : nv, b2v);
#pragma unroll
            for (int e = 0; e < 4; ++e) bslow[b][g][e] = bv[e] + b2v[e];
        }

    // prologue: B stage 0, A stage 0 and, with three B buffers, B stage 1
    static_for<FM>([&](auto i) __attribute__((always_inline)) { issue_b(0, 0, i); });
    static_for<FM>([&](auto i) __attribute__((always_inline)) { issue_a(0, 0, i); });
    if constexpr (NB == 3) static_for<FM>([&](auto i) __attribute__((always_inline)) { issue_b(1, 1, i); });

    f32x16 acc[FM][FN];
#pragma unroll
    for (int b = 0; b < FN; ++b)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int n = n0 + wn * TN + b * 32 + g * 8 + lhalf * 4;
            const bool fast = n + 4 <= n_hi;
            float bv[4], b2v[4];
            unpack4<T>(rb[b][g], bv);
            unpack4<T>(rb2[b][g], b2v);
#pragma unroll
            for (int a = 0; a < FM; ++a)
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[a][b][4 * g + e] = fast ? bv[e] + b2v[e] : bslow[b][g][e];
        }

    // LDS byte offset of this lane's fragment (row l % 32 of a 32-row group, k chunk 2 kk + l / 32
    // of the stage) for k step kk, within stage buffer 0 of A (fa) and of B (fb), for the wave's
    // first rows; fragment a (b) of the wave sits 32 a (32 b) rows = 4 KB further
    const unsigned ldsa0 = static_cast<unsigned>(reinterpret_cast<size_t>((lds_ptr_t)ldsA));
    const unsigned ldsb0 = static_cast<unsigned>(reinterpret_cast<size_t>((lds_ptr_t)ldsB));
    unsigned fa[4], fb[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        const unsigned f = ((lrow >> 3) * 64 + (lrow & 7) * 8 + ((2 * kk + lhalf) ^ (lrow & 7))) * 16;
        fa[kk] = ldsa0 + f + ((wm * TM) >> 3) * 1024;
        fb[kk] = ldsb0 + f + ((wn * TN) >> 3) * 1024;
    }
    // One k step: the MFMAs on fragments (ma, mb), row of tiles by row, each row preceded by
    // the reads of another k step's fragments a and b (into ra, rb, from LDS at ra_base,
    // rb_base) and, when kt >= 0, by load slots: rows 0 and 1 load A stage kt + 1 into A buffer
    // (kt + 1) % 2, rows 2 and 3 load B stage kt + NB - 1 into B buffer (kt + NB - 1) % NB (the
    // B loads go out last, so that a wait for all but them covers the A loads).  Nothing is
    // scheduled across the rows.
    auto step = [&](u32x4 (&ma)[FM], u32x4 (&mb)[FN], unsigned ra_base, unsigned rb_base, u32x4 (&ra)[FM],
                    u32x4 (&rb)[FN], int kt, int bbuf_next) __attribute__((always_inline)) {
        static_for<FM>([&](auto a) __attribute__((always_inline)) {
            ra[a] = lds_read16_at<a * 4096>(ra_base);
            rb[a] = lds_read16_at<a * 4096>(rb_base);
            if (kt >= 0) {
                if constexpr (a < 2)
                    issue_a(kt + 1, (kt + 1) & 1, 2 * a), issue_a(kt + 1, (kt + 1) & 1, 2 * a + 1);
                else
                    issue_b(kt + NB - 1, bbuf_next, 2 * (a - 2)), issue_b(kt + NB - 1, bbuf_next, 2 * (a - 2) + 1);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int b = 0; b < FN; ++b)
                acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, mb[b]),
                                                                    __builtin_bit_cast(bf16x8, ma[a]), acc[a][b], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        });
    };
    auto read_all = [&](unsigned ra_base, unsigned rb_base, u32x4 (&ra)[FM], u32x4 (&rb)[FN]) __attribute__((always_inline)) {
        static_for<FM>([&](auto a) __attribute__((always_inline)) {
            ra[a] = lds_read16_at<a * 4096>(ra_base);
            rb[a] = lds_read16_at<a * 4096>(rb_base);
        });
    };
    auto pin_all = [&](u32x4 (&af)[FM], u32x4 (&bf)[FN]) __attribute__((always_inline)) {
#pragma unroll
        for (int a = 0; a < FM; ++a) pin(af[a]);
#pragma unroll
        for (int b = 0; b < FN; ++b) pin(bf[b]);
    };
    // wait until this wave's loads of A stage st and B stage st have landed: with three B
    // buffers the eight B loads issued last (B stage st + 1) may still be in flight
    auto wait_stage = [&]() __attribute__((always_inline)) {
        if constexpr (NB == 3)
            asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
        else
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    };

    // Stage st sits in A buffer st % 2 and B buffer st % NB.  Iteration st: wait for it, barrier
    // (every wave's share has landed; stage st - 1 is fully read), then four k steps; step kk
    // multiplies the fragments of the step before it (step 3 of stage st - 1 for kk = 0) while it
    // reads its own, and step 0 also loads A stage st + 1 and B stage st + NB - 1.
    u32x4 f0a[FM], f0b[FN], f1a[FM], f1b[FN];
    wait_stage();
    __builtin_amdgcn_s_barrier();
    read_all(fa[0], fb[0], f0a, f0b);
    lds_wait();
    pin_all(f0a, f0b);
    step(f0a, f0b, fa[1], fb[1], f1a, f1b, 0, (NB - 1) % NB);
    lds_wait();
    pin_all(f1a, f1b);
    step(f1a, f1b, fa[2], fb[2], f0a, f0b, -1, 0);
    lds_wait();
    pin_all(f0a, f0b);
    step(f0a, f0b, fa[3], fb[3], f1a, f1b, -1, 0);
    lds_wait();
    pin_all(f1a, f1b);
    int bcur = 0;                                      // B buffer of stage st
    for (int st = 1; st < nk; ++st) {
        bcur = bcur == NB - 1 ? 0 : bcur + 1;
        const int bnext = bcur == 0 ? NB - 1 : bcur - 1;   // (st + NB - 1) % NB: stage st - 1's buffer
        const unsigned abase = (st & 1) * SA * 16, bbase = bcur * SB * 16;
        wait_stage();                                  // this wave's share of stage st has landed
        __builtin_amdgcn_s_barrier();                  // every wave's has; stage st - 1 fully read
        step(f1a, f1b, abase + fa[0], bbase + fb[0], f0a, f0b, st, bnext);
        lds_wait();
        pin_all(f0a, f0b);
        step(f0a, f0b, abase + fa[1], bbase + fb[1], f1a, f1b, -1, 0);
        lds_wait();
        pin_all(f1a, f1b);
        step(f1a, f1b, abase + fa[2], bbase + fb[2], f0a, f0b, -1, 0);
        lds_wait();
        pin_all(f0a, f0b);
        step(f0a, f0b, abase + fa[3], bbase + fb[3], f1a, f1b, -1, 0);
        lds_wait();
        pin_all(f1a, f1b);
    }
#pragma unroll
    for (int a = 0; a < FM; ++a)
#pragma unroll
        for (int b = 0; b < FN; ++b)
            acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, f1b[b]),
                                                                __builtin_bit_cast(bf16x8, f1a[a]), acc[a][b], 0, 0, 0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // the last (unread) loads land before LDS is reused

    // --- epilogue ---------------------------------------------------------------------------
    // Without a residual and with a bf16 output, v = act(acc) is rounded in the MFMA layout and
    // the bf16 tile is staged in LDS in one pass; otherwise the float32 sums are staged in two
    // passes of 128 rows and finished in 8-column chunks as gemm_kernel finishes them (residual,
    // activation, rounding).  Either way the stores are whole 16-byte chunks along rows, and a
    // pass reads all its residual chunks before its first store, so that no wait in the epilogue
    // waits for a store.
    __syncthreads();                                   // every wave is done with the operand stages
    unsigned char* tile = reinterpret_cast<unsigned char*>(lds);
    const int tid = threadIdx.x;
    const T* resp = static_cast<const T*>(p.res);
    if (!resp && !p.out_f32) {
        // (one copy of the unrolled tile per activation: a per-element choice would evaluate
        // every activation for all 256 values)
        auto stage_bf16 = [&](auto act) __attribute__((always_inline)) {
            static_for<FM>([&](auto a) __attribute__((always_inline)) {
                static_for<FN>([&](auto b) __attribute__((always_inline)) {
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        float v[4];
#pragma unroll
                        for (int e = 0; e < 4; ++e) v[e] = act_f(acc_read(acc[a][b][4 * g + e]) + 0.0f, decltype(act)::value);
                        const int row = wm * TM + a * 32 + lrow, col = wn * TN + b * 32 + g * 8 + lhalf * 4;
                        *reinterpret_cast<bf16x4*>(tile + row * kWideRowB + col * 2) =
                            bf16x4{(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
                    }
                    // one tile at a time: the accumulators are read out only when they are used
                    __builtin_amdgcn_sched_barrier(0);
                });
            });
        };
        if (p.act == MOPAR_ACT_RELU)
            stage_bf16(std::integral_constant<int, MOPAR_ACT_RELU>{});
        else if (p.act == MOPAR_ACT_GELU)
            stage_bf16(std::integral_constant<int, MOPAR_ACT_GELU>{});
        else
            stage_bf16(std::integral_constant<int, MOPAR_ACT_NONE>{});
        __syncthreads();
        T* C = static_cast<T*>(p.C);
        for (int i = 0; i < BM / 8; ++i) {
            const int r = i * 8 + (tid >> 5), c = (tid & 31) * 8;
            const int m = m0 + r, n = n0 + c;
            if (m >= Mi || n >= n_hi) continue;
            const uint4 w = *reinterpret_cast<const uint4*>(tile + r * kWideRowB + c * 2);
            T* dst = C + static_cast<int64_t>(m) * p.ldc + n;
            const int nv = min(8, n_hi - n);
            if (nv == 8 && aligned16(dst)) {
                *reinterpret_cast<uint4*>(dst) = w;
            } else {
                const unsigned short* h = reinterpret_cast<const unsigned short*>(&w);
                for (int e = 0; e < nv; ++e) reinterpret_cast<unsigned short*>(dst)[e] = h[e];
            }
        }
        return;
    }
    constexpr int NCH = TM * BN / 8 / 256;             // 8-column chunks per thread and pass
    const int cc = tid & 31, cr = tid >> 5;            // chunk column; first row (then every 8th)
    const int c0 = n0 + cc * 8;
    const int cval = max(0, min(8, n_hi - c0));
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        if (h) __syncthreads();                        // the first half's rows are all read
        if (wm == h) {
            static_for<FM>([&](auto a) __attribute__((always_inline)) {
                static_for<FN>([&](auto b) __attribute__((always_inline)) {
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int row = a * 32 + lrow, col = wn * TN + b * 32 + g * 8 + lhalf * 4;
                        *reinterpret_cast<f32x4*>(tile + row * kWideRowF + col * 4) =
                            f32x4{acc_read(acc[a][b][4 * g]), acc_read(acc[a][b][4 * g + 1]),
                                  acc_read(acc[a][b][4 * g + 2]), acc_read(acc[a][b][4 * g + 3])};
                    }
                    __builtin_amdgcn_sched_barrier(0);
                });
            });
        }
        __syncthreads();
        Raw8<T> rraw[NCH];
        bool rfast[NCH];
        if (resp) {
#pragma unroll
            for (int i = 0; i < NCH; ++i) {
                const int m = m0 + h * TM + cr + 8 * i;
                const int64_t idx = static_cast<int64_t>(m) * p.ldc + c0;
                rfast[i] = m < Mi && cval == 8 && aligned16(resp + idx);
                rraw[i] = load_raw8<T>(rfast[i] ? resp + idx : nullptr, kZeroChunk);
            }
        }
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int r = cr + 8 * i;
            const int m = m0 + h * TM + r;
            if (m >= Mi || cval == 0) continue;
            float v[8], rsd[8];
            const f32x4 lo = *reinterpret_cast<const f32x4*>(tile + r * kWideRowF + cc * 32);
            const f32x4 hi = *reinterpret_cast<const f32x4*>(tile + r * kWideRowF + cc * 32 + 16);
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = lo[e], v[4 + e] = hi[e];
            const int64_t idx = static_cast<int64_t>(m) * p.ldc + c0;
            if (resp && rfast[i])
                unpack8<T>(rraw[i], rsd);
            else
                load8<T>(resp, idx, resp ? cval : 0, rsd);
            if (p.act == MOPAR_ACT_NONE) {
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = v[e] + rsd[e];
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] = act_f(v[e] + rsd[e], p.act);
            }
            if (p.out_f32)
                store8<float>(static_cast<float*>(p.C), idx, v, cval);
            else
                store8<T>(static_cast<T*>(p.C), idx, v, cval);
        }
    }
}

// Persistent form of gemm_wide_kernel, used when the launch brings tile counters (one word per
// XCD, zeroed by the launcher before the launch): one block per CU, fed from a queue.  The blocks
// of XCD x take x's run of tiles, first one each by block index, then from x's counter, so that a
// block whose CU is busy with another stream's kernel when the launch starts takes fewer tiles,
// and the blocks an XCD runs together still work on neighbouring tiles.  Per tile the MFMA
// arithmetic is gemm_wide_kernel's.  What changes is the hand-over between tiles: the next
// tile's number is fetched while the current tile's first stage runs, its first stage is loaded
// during the current tile's last stage, its bias while the current tile is stored, and the
// epilogue stores straight from the accumulators (one store per group of four columns, an
// out-of-range offset for the groups that are not written, so that every tile issues the same
// number of stores and the next tile waits for its first stage without waiting for them).  It
// takes products without a residual or an activation (the others run on gemm_wide_kernel).
__global__ __launch_bounds__(256, 1) void gemm_wide_persistent(const GemmParams p) {
    using T = __bf16;
    constexpr int BM = 256, BN = 256, TM = 128, TN = 128;
    constexpr int FM = TM / 32, FN = TN / 32;
    constexpr int NBA = BM / 8, NBB = BN / 8;
    constexpr int NW = 4;
    constexpr int LA = NBA / NW, LB = NBB / NW;
    constexpr int SA = NBA * 64, SB = NBB * 64;
    constexpr int BK = 64;
    constexpr int NSTORE = FM * FN * 4;          // stores per lane and tile (regular tiles)
    static_assert(LA == LB && LA == 2 * FM, "two load slots per row of fragments");
    static_assert(NSTORE == 64, "the first-stage wait below lets 63 stores stay in flight");
    __shared__ uint4 lds[2 * SA + 2 * SB];
    __shared__ int s_ticket;
    __shared__ __attribute__((aligned(16))) float s_bias[BN];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int lrow = lane & 31, lhalf = lane >> 5;
    touch_kernargs<sizeof(GemmParams)>();

    const int xcd = blockIdx.x & 7, gx = static_cast<int>(gridDim.x >> 3);
    const int t_lo = xcd * p.g_per_xcd;
    const int cx = min(p.g_per_xcd, p.g_total - t_lo);   // tiles of this XCD's run
    unsigned* const ctr = p.wide_ctr + xcd;
    const int Mi = static_cast<int>(p.M);
    const int nk = p.g_nk;                               // >= 2 (checked at launch)
    const int ktail = (p.K % BK) ? nk - 1 : nk;
    const int cl = (lane & 7) ^ (lane >> 3);

    // tile li of this XCD's run -> rows m0.., columns n0 .. n_hi - 1; false when the tile lies
    // past a narrower sub-slice's last column
    auto decode = [&](int li, int& m0, int& n0, int& n_hi) __attribute__((always_inline)) -> bool {
        const unsigned t = static_cast<unsigned>(t_lo + li);
        constexpr int GM = kWideGroupM;
        const unsigned group = p.g_div_group.div(t);
        const unsigned within = t - group * static_cast<unsigned>(GM * p.g_cols);
        const bool last = static_cast<int>(group) == (p.g_mt - 1) / GM;
        const unsigned gm = last ? static_cast<unsigned>(p.g_mt - group * GM) : GM;
        const unsigned colu = last ? p.g_div_last.div(within) : within / GM;
        const int mti = static_cast<int>(group * GM + (within - colu * gm));
        const unsigned c1 = p.g_div_nt.div(colu);
        const int nti = static_cast<int>(colu - c1 * static_cast<unsigned>(p.g_nt));
        const int j = static_cast<int>(c1);
        const int n_lo = j * p.g_q + min(j, p.g_rr);
        n_hi = (j + 1) * p.g_q + min(j + 1, p.g_rr);
        n0 = n_lo + nti * BN;
        m0 = mti * BM;
        return n0 < n_hi;
    };
    // one more tile number from the queue, the same for every thread of the block
    auto fetch_now = [&]() __attribute__((always_inline)) -> int {
        if (threadIdx.x == 0) s_ticket = gx + static_cast<int>(__hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
        __syncthreads();
        const int v = __builtin_amdgcn_readfirstlane(s_ticket);
        __syncthreads();
        return v;
    };
    auto offsets = [&](int m0, int n0, int n_hi, unsigned (&va)[LA], unsigned (&vb)[LB]) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < LA; ++i) {
            const int m = m0 + (wave + NW * i) * 8 + (lane >> 3);
            const int mc = m < Mi ? m : Mi - 1;
            va[i] = static_cast<unsigned>(mc) * static_cast<unsigned>(p.lda * sizeof(T)) + static_cast<unsigned>(cl * 16);
        }
#pragma unroll
        for (int i = 0; i < LB; ++i) {
            const int n = n0 + (wave + NW * i) * 8 + (lane >> 3);
            const int nc = n < n_hi ? n : n_hi - 1;
            vb[i] = static_cast<unsigned>(nc) * static_cast<unsigned>(p.K * sizeof(T)) + static_cast<unsigned>(cl * 16);
        }
    };
    uint4* const ldsA = &lds[0];
    uint4* const ldsB = &lds[2 * SA];
    // Load slot s2 of one operand's stage kt (clamped to the last stage) into buffer buf.  (Issuing
    // one of these 1 KB loads holds the wave for ~50 cycles, measured; the K loop puts one after
    // every second MFMA, so that the MFMAs already issued keep the matrix unit busy meanwhile.)
    auto load_a = [&](const unsigned (&va)[LA], int kt, int buf, int s2) __attribute__((always_inline)) {
        kt = __builtin_amdgcn_readfirstlane(kt < nk ? kt : nk - 1);
        const unsigned soff = static_cast<unsigned>(kt) * (BK * sizeof(T));
        const bool kin = kt != ktail || kt * BK + cl * 8 < p.K;
        // (the offset is settled before the load: a branch around the load would turn the
        // scalar offset into a per-lane one, which the compiler then loops over)
        unsigned v = kin ? va[s2] : kOOB;
        asm volatile("" : "+v"(v));
        buffer_load_lds(p.A, p.a_bytes, (lds_ptr_t)(ldsA + buf * SA + (wave + NW * s2) * 64), v, soff);
    };
    auto load_b = [&](const unsigned (&vb)[LB], int kt, int buf, int s2) __attribute__((always_inline)) {
        kt = __builtin_amdgcn_readfirstlane(kt < nk ? kt : nk - 1);
        const unsigned soff = static_cast<unsigned>(kt) * (BK * sizeof(T));
        const bool kin = kt != ktail || kt * BK + cl * 8 < p.K;
        // (the offset is settled before the load: a branch around the load would turn the
        // scalar offset into a per-lane one, which the compiler then loops over)
        unsigned v = kin ? vb[s2] : kOOB;
        asm volatile("" : "+v"(v));
        buffer_load_lds(p.B, p.b_bytes, (lds_ptr_t)(ldsB + buf * SB + (wave + NW * s2) * 64), v, soff);
    };
    // Bias + second bias of a tile: thread t reads column n0 + t (zero past n_hi) and the sums go
    // through LDS (s_bias), from which every wave starts its accumulators -- the same float
    // additions as gemm_kernel's, per column.
    const T* biasp = static_cast<const T*>(p.bias);
    const T* bias2p = static_cast<const T*>(p.bias2);
    auto bias_col = [&](int n0, int n_hi, float& bv, float& b2v) __attribute__((always_inline)) {
        const int n = n0 + static_cast<int>(threadIdx.x);
        bv = (biasp && n < n_hi) ? ld_f(biasp, n) : 0.0f;
        b2v = (bias2p && n < n_hi) ? ld_f(bias2p, n) : 0.0f;
    };
    f32x16 acc[FM][FN];
    auto bias_init = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int b = 0; b < FN; ++b)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const f32x4 bsum = *reinterpret_cast<const f32x4*>(&s_bias[wn * TN + b * 32 + g * 8 + lhalf * 4]);
#pragma unroll
                for (int a = 0; a < FM; ++a)
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[a][b][4 * g + e] = bsum[e];
            }
    };

    const unsigned ldsa0 = static_cast<unsigned>(reinterpret_cast<size_t>((lds_ptr_t)ldsA));
    const unsigned ldsb0 = static_cast<unsigned>(reinterpret_cast<size_t>((lds_ptr_t)ldsB));
    unsigned fa[4], fb[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        const unsigned f = ((lrow >> 3) * 64 + (lrow & 7) * 8 + ((2 * kk + lhalf) ^ (lrow & 7))) * 16;
        fa[kk] = ldsa0 + f + ((wm * TM) >> 3) * 1024;
        fb[kk] = ldsb0 + f + ((wn * TN) >> 3) * 1024;
    }
    // One k step: MFMAs on (ma, mb) row by row, each row preceded by the reads of the next k step's
    // fragments; loads(2 a + h) after the row's MFMA 2 h + 1.  Nothing is scheduled across.
    auto step = [&](u32x4 (&ma)[FM], u32x4 (&mb)[FN], unsigned ra_base, unsigned rb_base, u32x4 (&ra)[FM],
                    u32x4 (&rb_)[FN], auto&& loads) __attribute__((always_inline)) {
        static_for<FM>([&](auto a) __attribute__((always_inline)) {
            ra[a] = lds_read16_at<a * 4096>(ra_base);
            rb_[a] = lds_read16_at<a * 4096>(rb_base);
            __builtin_amdgcn_sched_barrier(0);
            static_for<FN>([&](auto b) __attribute__((always_inline)) {
                acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, mb[b]),
                                                                    __builtin_bit_cast(bf16x8, ma[a]), acc[a][b], 0, 0, 0);
                if constexpr (b % 2 == 1) loads(2 * a + b / 2);
                __builtin_amdgcn_sched_barrier(0);
            });
        });
    };
    auto no_loads = [](int) __attribute__((always_inline)) {};
    auto pin_all = [&](u32x4 (&af)[FM], u32x4 (&bf)[FN]) __attribute__((always_inline)) {
#pragma unroll
        for (int a = 0; a < FM; ++a) pin(af[a]);
#pragma unroll
        for (int b = 0; b < FN; ++b) pin(bf[b]);
    };

    // --- first tile -------------------------------------------------------------------------
    int li = static_cast<int>(blockIdx.x >> 3);
    int m0 = 0, n0 = 0, n_hi = 0;
    for (;;) {                                          // (block-uniform)
        if (li >= cx) return;
        if (decode(li, m0, n0, n_hi)) break;
        li = fetch_now();
    }
    unsigned va[LA], vb[LB];
    offsets(m0, n0, n_hi, va, vb);
    int par = 0;                                        // stage s of the tile sits in buffers (par + s) & 1
    {
        float bv, b2v;
        bias_col(n0, n_hi, bv, b2v);
        s_bias[threadIdx.x] = bv + b2v;
    }
#pragma unroll
    for (int s2 = 0; s2 < LB; ++s2) load_b(vb, 0, 0, s2);
#pragma unroll
    for (int s2 = 0; s2 < LA; ++s2) load_a(va, 0, 0, s2);
    bool wait_all = true;                               // the first stage's loads are the newest in flight

    const uint32_t esz = p.out_f32 ? 4u : 2u;
    const __amdgpu_buffer_rsrc_t crs = __builtin_amdgcn_make_buffer_rsrc(p.C, static_cast<short>(0),
                                                                         static_cast<int>(p.c_bytes), kRsrcWord3);
    const bool c_aligned = (reinterpret_cast<uintptr_t>(p.C) & (4 * esz - 1)) == 0 && (p.ldc & 3) == 0;

    for (;;) {
        u32x4 f0a[FM], f0b[FN], f1a[FM], f1b[FN];
        int li_next = cx;                               // the next tile (>= cx: none)
        int m0n = 0, n0n = 0, n_hin = 0;
        bool next_ok = false;
        unsigned van[LA], vbn[LB];
        int ticket_v = 0;
        float nbv = 0.0f, nb2v = 0.0f;                  // the next tile's bias column
        auto take_ticket = [&]() __attribute__((always_inline)) {
            // (the ticket's load was issued in stage 0; this wait is the stage wait's)
            if (threadIdx.x == 0) s_ticket = ticket_v;
        };
        auto read_ticket = [&]() __attribute__((always_inline)) {
            li_next = __builtin_amdgcn_readfirstlane(s_ticket);
            // (uniform values, kept in scalar registers: otherwise the compiler may treat the
            // branches on them as divergent and loop over the loads' scalar offsets)
            next_ok = __builtin_amdgcn_readfirstlane((li_next < cx && decode(li_next, m0n, n0n, n_hin)) ? 1 : 0) != 0;
            m0n = __builtin_amdgcn_readfirstlane(m0n);
            n0n = __builtin_amdgcn_readfirstlane(n0n);
            n_hin = __builtin_amdgcn_readfirstlane(n_hin);
            if (next_ok) offsets(m0n, n0n, n_hin, van, vbn);
        };

        // stage 0
        if (wait_all)
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        else
            asm volatile("s_waitcnt vmcnt(63)" ::: "memory");
        __builtin_amdgcn_s_barrier();                  // (also: s_bias holds this tile's bias)
        bias_init();
        {
            const unsigned ab = (par & 1) * SA * 16, bb = (par & 1) * SB * 16;
            const int nb = (par + 1) & 1;
            if (threadIdx.x == 0)
                ticket_v = gx + static_cast<int>(__hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
            static_for<FM>([&](auto a) __attribute__((always_inline)) {
                f0a[a] = lds_read16_at<a * 4096>(ab + fa[0]);
                f0b[a] = lds_read16_at<a * 4096>(bb + fb[0]);
            });
            lds_wait();
            pin_all(f0a, f0b);
            auto ld1b = [&](int s2) __attribute__((always_inline)) { load_b(vb, 1, nb, s2); };
            auto ld1a = [&](int s2) __attribute__((always_inline)) { load_a(va, 1, nb, s2); };
            step(f0a, f0b, ab + fa[1], bb + fb[1], f1a, f1b, ld1b);
            lds_wait();
            pin_all(f1a, f1b);
            step(f1a, f1b, ab + fa[2], bb + fb[2], f0a, f0b, ld1a);
            lds_wait();
            pin_all(f0a, f0b);
            step(f0a, f0b, ab + fa[3], bb + fb[3], f1a, f1b, no_loads);
            lds_wait();
            pin_all(f1a, f1b);
        }
        // stages 1 .. nk - 2: this tile's next stage
        for (int st = 1; st < nk - 1; ++st) {
            const int buf = (par + st) & 1;
            const unsigned ab = buf * SA * 16, bb = buf * SB * 16;
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            if (st == 1) take_ticket();
            __builtin_amdgcn_s_barrier();
            if (st == 1) read_ticket();
            auto ldnb = [&](int s2) __attribute__((always_inline)) { load_b(vb, st + 1, buf ^ 1, s2); };
            auto ldna = [&](int s2) __attribute__((always_inline)) { load_a(va, st + 1, buf ^ 1, s2); };
            step(f1a, f1b, ab + fa[0], bb + fb[0], f0a, f0b, ldnb);
            lds_wait();
            pin_all(f0a, f0b);
            step(f0a, f0b, ab + fa[1], bb + fb[1], f1a, f1b, ldna);
            lds_wait();
            pin_all(f1a, f1b);
            step(f1a, f1b, ab + fa[2], bb + fb[2], f0a, f0b, no_loads);
            lds_wait();
            pin_all(f0a, f0b);
            step(f0a, f0b, ab + fa[3], bb + fb[3], f1a, f1b, no_loads);
            lds_wait();
            pin_all(f1a, f1b);
        }
        // last stage: the next tile's first stage (or, without one, this stage again, unread)
        {
            const int buf = (par + nk - 1) & 1;
            const unsigned ab = buf * SA * 16, bb = buf * SB * 16;
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            if (nk == 2) take_ticket();
            __builtin_amdgcn_s_barrier();
            if (nk == 2) read_ticket();
            if (next_ok) bias_col(n0n, n_hin, nbv, nb2v);  // used in the epilogue
            auto ldxb = [&](int s2) __attribute__((always_inline)) {
                if (next_ok) load_b(vbn, 0, buf ^ 1, s2); else load_b(vb, nk - 1, buf ^ 1, s2);
            };
            auto ldxa = [&](int s2) __attribute__((always_inline)) {
                if (next_ok) load_a(van, 0, buf ^ 1, s2); else load_a(va, nk - 1, buf ^ 1, s2);
            };
            step(f1a, f1b, ab + fa[0], bb + fb[0], f0a, f0b, ldxb);
            lds_wait();
            pin_all(f0a, f0b);
            step(f0a, f0b, ab + fa[1], bb + fb[1], f1a, f1b, ldxa);
            lds_wait();
            pin_all(f1a, f1b);
            step(f1a, f1b, ab + fa[2], bb + fb[2], f0a, f0b, no_loads);
            lds_wait();
            pin_all(f0a, f0b);
            step(f0a, f0b, ab + fa[3], bb + fb[3], f1a, f1b, no_loads);
            lds_wait();
            pin_all(f1a, f1b);
        }
#pragma unroll
        for (int a = 0; a < FM; ++a)
#pragma unroll
            for (int b = 0; b < FN; ++b)
                acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, f1b[b]),
                                                                    __builtin_bit_cast(bf16x8, f1a[a]), acc[a][b], 0, 0, 0);

        // --- epilogue of this tile ---------------------------------------------------------
        // (every wave has read the bias of this tile long ago: s_bias takes the next one's)
        if (next_ok) s_bias[threadIdx.x] = nbv + nb2v;
        // a tile is regular when every group of four columns is whole or absent and aligned:
        // then one 8-byte (bf16) or 16-byte (float32) store per group, else one per element
        const bool regular = c_aligned && (n0 & 3) == 0 && (n_hi & 3) == 0;
        static_for<FM>([&](auto a) __attribute__((always_inline)) {
            static_for<FN>([&](auto b) __attribute__((always_inline)) {
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int m = m0 + wm * TM + a * 32 + lrow;
                    const int n = n0 + wn * TN + b * 32 + g * 8 + lhalf * 4;
                    const int nv = m < Mi ? max(0, min(4, n_hi - n)) : 0;
                    const unsigned off = (static_cast<unsigned>(m) * static_cast<unsigned>(p.ldc) + static_cast<unsigned>(n)) * esz;
                    float v[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = acc_read(acc[a][b][4 * g + e]) + 0.0f;
                    if (regular) {
                        const unsigned o = nv == 4 ? off : kOOB;
                        if (p.out_f32) {
                            __builtin_amdgcn_raw_buffer_store_b128(u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]),
                                                                         __float_as_uint(v[2]), __float_as_uint(v[3])},
                                                                   crs, static_cast<int>(o), 0, 0);
                        } else {
                            const bf16x4 h = {(__bf16)v[0], (__bf16)v[1], (__bf16)v[2], (__bf16)v[3]};
                            __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, h), crs, static_cast<int>(o), 0, 0);
                        }
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const unsigned o = e < nv ? off + e * esz : kOOB;
                            if (p.out_f32)
                                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v[e]), crs, static_cast<int>(o), 0, 0);
                            else
                                __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, (__bf16)v[e]),
                                                                      crs, static_cast<int>(o), 0, 0);
                        }
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            });
        });

        // --- the next tile -------------------------------------------------------------------
        if (next_ok) {
            m0 = m0n, n0 = n0n, n_hi = n_hin;
#pragma unroll
            for (int i = 0; i < LA; ++i) va[i] = van[i], vb[i] = vbn[i];
            par = (par + nk) & 1;
            // its first stage went out before this tile's 64 stores (irregular tiles issue more)
            wait_all = !regular;
            continue;
        }
        // no prefetched tile: take numbers until one is not empty (or the run is done)
        li = li_next;
        for (;;) {
            if (li >= cx) return;
            if (decode(li, m0, n0, n_hi)) break;
            li = fetch_now();
        }
        offsets(m0, n0, n_hi, va, vb);
        par = 0;
        __syncthreads();                                // every wave is done with both buffers
        {
            float bv, b2v;
            bias_col(n0, n_hi, bv, b2v);
            s_bias[threadIdx.x] = bv + b2v;
        }
#pragma unroll
        for (int s2 = 0; s2 < LB; ++s2) load_b(vb, 0, 0, s2);
#pragma unroll
        for (int s2 = 0; s2 < LA; ++s2) load_a(va, 0, 0, s2);
        wait_all = true;
    }
}

// Split-K finish: sum the partials in split order, then the usual epilogue.
template <typename T>
__global__ void splitk_reduce_kernel(const GemmParams p) {
    touch_kernargs<sizeof(GemmParams)>();
    // one thread per 4 columns of a row; M * ceil(N / 4) < 2^31 (checked at launch)
    const unsigned groups = static_cast<unsigned>(p.N + 3) / 4;
    const unsigned t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= static_cast<unsigned>(p.M) * groups) return;
    const unsigned mu = p.r_div_groups.div(t);
    const int64_t m = mu;
    const int n = static_cast<int>(t - mu * groups) * 4;
    const int nvalid = min(4, p.N - n);
    // bias, second bias and residual go out first, so their latency overlaps the partials'
    float bias[4] = {0.f, 0.f, 0.f, 0.f}, bias2[4] = {0.f, 0.f, 0.f, 0.f}, rsd[4] = {0.f, 0.f, 0.f, 0.f};
    if (p.bias) ld4(static_cast<const T*>(p.bias), n, nvalid, bias);
    if (p.bias2) ld4(static_cast<const T*>(p.bias2), n, nvalid, bias2);
    if (p.res) ld4(static_cast<const T*>(p.res), m * p.ldc + n, nvalid, rsd);
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    const int64_t plane = p.M * static_cast<int64_t>(p.N);
    const float* src = p.partial + m * p.N + n;
    if (nvalid == 4 && (p.N & 3) == 0) {
        f32x4 part[16];                       // splits <= 16: all loads in flight together
#pragma unroll
        for (int s = 0; s < 16; ++s)
            if (s < p.splits) part[s] = *reinterpret_cast<const f32x4*>(src + s * plane);
#pragma unroll
        for (int s = 0; s < 16; ++s)
            if (s < p.splits)
                for (int e = 0; e < 4; ++e) v[e] += part[s][e];
    } else {
        for (int s = 0; s < p.splits; ++s)
            for (int e = 0; e < nvalid; ++e) v[e] += src[s * plane + e];
    }
    for (int q = 0; q < 4; ++q) v[q] = act_f((v[q] + (bias[q] + bias2[q])) + rsd[q], p.act);
    const int64_t idx = m * p.ldc + n;
    if (p.out_f32)
        store4<float>(static_cast<float*>(p.C), idx, v, nvalid);
    else
        store4<T>(static_cast<T*>(p.C), idx, v, nvalid);
}

// ---------------------------------------------------------------------------
// 3x3 convolutions (stride 1, padding 1) over bf16 images of 64 to 512 channels
// (multiples of 64) and at most 56 x 56 pixels, patch-staged.  The implicit
// GEMM above fetches every input pixel once per tap (nine times); here a block
// owns a TH x 8 tile of output pixels of one image (8 x 8 in use) and BN output
// channels of one sub-slice, and for each 64-channel chunk it stages the
// (TH + 2) x 10 input patch around its tile (one pixel of halo each way, zeros
// outside the image) once, with the nine taps' weight rows, then forms all nine
// taps' A fragments from that patch in LDS (about a sixth of the A bytes; the
// win is largest on narrow sub-slices, whose A traffic dominates).  Images of
// more than two chunks take two chunk buffers, the next chunk's loads going out
// before the current chunk's products (64 KB of LDS per block; with fewer chunks
// one buffer, which leaves room for more resident blocks: measured faster on
// ResNet-50's stages 1 and 2, 7.7-8.9 us against 10.8-14.1 us).  Loads use the same whole-line, XOR-swizzled layout as
// above (patch pixels and weight rows in place of tile rows).  The k order is
// chunk, then tap, then the two 32-wide steps; it depends only on the op, not
// on BN, TH or the sub-slice, so sub-sliced and unsplit launches agree bit for
// bit.  TH / 2 waves each take two tile rows (16 pixels) by BN columns; the
// accumulators start at the bias and the epilogue stores from the MFMA layout
// (residual, activation).
// ---------------------------------------------------------------------------
constexpr int HTW = 8;                       // output tile width; its height TH is a parameter

bool conv_halo_ok(int dtype, int kh, int kw, int stride, int pad, int cs, int n_out, int out_h, int out_w, int64_t m) {
    // Small convs only: at most 2^31 multiply-adds (M x N x K; each of ResNet-50's stride-1 3x3
    // convs at batch 8 is 0.92 G).  On those the implicit GEMM's large tiles leave CUs idle or
    // need split-K and a second launch, and this kernel is faster (stages 3 and 4: 9.0-10.0
    // against 13.5-16.6 us and 12.1-12.2 against 14.6-15.2 us).  On larger convs the patch,
    // re-read for every 16 output channels, and the small tiles lose to the GEMM, measured:
    // VGG-16 at batch 16, 7.4-29.6 G multiply-adds, 51-192 us here against 36-74 us; and over
    // images above 56 x 56.
    if (!(dtype == MOPAR_BF16 && kh == 3 && kw == 3 && stride == 1 && pad == 1 && cs % 64 == 0 && cs <= 512 &&
          n_out >= 1 && n_out <= 512 && out_h >= 7 && out_w >= 7 && int64_t(out_h) * out_w <= 56 * 56 && m >= 0 &&
          m < (int64_t(1) << 31)))
        return false;
    // (the checks above bound the product below 2^53)
    return m * n_out * (int64_t(kh) * kw * cs) <= (int64_t(1) << 31);
}

template <int BN, int TH, int NBUF>
__global__ __launch_bounds__(TH * HTW / 16 * 64) void conv3_halo_kernel(const GemmParams p) {
    using T = __bf16;
    constexpr int NW = TH * HTW / 16;           // waves: 16 tile pixels (two tile rows) each
    constexpr int PW = HTW + 2, PIX = (TH + 2) * PW;   // patch width, pixels
    constexpr int HPBLK = (PIX + 7) / 8;        // patch load blocks of 8 pixels
    constexpr int FN = BN / 16;
    constexpr int BPT = BN / 8;                 // weight load blocks per tap
    constexpr int NBB = 9 * BPT;                // weight load blocks per chunk
    constexpr int LP = (HPBLK + NW - 1) / NW, LB = (NBB + NW - 1) / NW;   // load slots per wave
    // NBUF chunk buffers: patch blocks, weight blocks and, with two buffers, one block for the
    // load slots past the last block (a wave whose share ends early still issues LP + LB loads,
    // of zeros, there, so that every wave's wait count is the same)
    static_assert(NBUF == 1 || NBUF == 2, "chunk buffers");
    constexpr int CHB = HPBLK + NBB + (NBUF == 2 ? 1 : 0);
    __shared__ uint4 lds[NBUF * CHB * 64];
    touch_kernargs<sizeof(GemmParams)>();
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

    // block -> (image, spatial tile, sub-slice, n tile); the blocks that share a patch are
    // consecutive, and each XCD runs a contiguous range of them
    const unsigned t = (blockIdx.x % 8) * static_cast<unsigned>(p.g_per_xcd) + blockIdx.x / 8;
    if (t >= static_cast<unsigned>(p.g_total)) return;
    const unsigned tile = p.g_div_group.div(t);
    const unsigned col = t - tile * static_cast<unsigned>(p.g_cols);
    const unsigned j = p.g_div_nt.div(col);
    const int nti = static_cast<int>(col - j * static_cast<unsigned>(p.g_nt));
    const unsigned img = p.h_div_tiles.div(tile);
    const unsigned tin = tile - img * static_cast<unsigned>(p.h_tiles);
    const unsigned tyi = p.h_div_tx.div(tin);
    const int oh0 = static_cast<int>(tyi) * TH, ow0 = static_cast<int>(tin - tyi * static_cast<unsigned>(p.h_tx)) * HTW;
    const int jj = static_cast<int>(j);
    const int n_lo = jj * p.g_q + min(jj, p.g_rr), n_hi = (jj + 1) * p.g_q + min(jj + 1, p.g_rr);
    const int n0 = n_lo + nti * BN;
    if (n0 >= n_hi) return;                     // block-uniform, before any barrier

    // loads of chunk q: patch block b covers pixels 8b .. 8b + 7 (pixel pp at patch row pp / 10,
    // column pp % 10), weight block b covers rows 8 (b % BPT) .. +7 of tap b / BPT; lane l takes
    // entity 8b + l / 8, chunk cl = (l % 8) ^ (l / 8); a chunk's byte offset adds 128 q
    const int cl = (lane & 7) ^ (lane >> 3);
    const unsigned pix_bytes = static_cast<unsigned>(p.cs) * 2u;
    unsigned voffP[LP], voffB[LB];
#pragma unroll
    for (int i = 0; i < LP; ++i) {
        const int pp = 8 * min(wave + NW * i, HPBLK - 1) + (lane >> 3);
        const int ih = oh0 - 1 + pp / PW, iw = ow0 - 1 + pp % PW;
        const bool in = pp < PIX && static_cast<unsigned>(ih) < static_cast<unsigned>(p.img_h) &&
                        static_cast<unsigned>(iw) < static_cast<unsigned>(p.img_w);
        voffP[i] = in ? (static_cast<unsigned>((static_cast<int>(img) * p.img_h + ih) * p.img_w + iw)) * pix_bytes +
                            static_cast<unsigned>(cl * 16)
                      : kOOB;
    }
#pragma unroll
    for (int i = 0; i < LB; ++i) {
        const int b = min(wave + NW * i, NBB - 1);
        const int tap = b / BPT, n = min(n0 + (b % BPT) * 8 + (lane >> 3), n_hi - 1);
        voffB[i] = static_cast<unsigned>(n) * static_cast<unsigned>(p.K * 2) + static_cast<unsigned>(tap) * pix_bytes +
                   static_cast<unsigned>(cl * 16);
    }

    // epilogue set-up (MFMA layout): this lane's tile pixel and four columns per n fragment
    const int pix = wave * 16 + (lane & 15);
    const int oh = oh0 + (pix >> 3), ow = ow0 + (pix & 7);
    const bool row_ok = oh < p.out_h && ow < p.out_w;
    const int64_t row = (static_cast<int64_t>(img) * p.out_h + oh) * p.out_w + ow;
    int ncol[FN], nval[FN];
    f32x4 acc[FN];
#pragma unroll
    for (int b = 0; b < FN; ++b) {
        ncol[b] = n0 + b * 16 + (lane >> 4) * 4;
        nval[b] = max(0, min(4, n_hi - ncol[b]));
        float bv[4], b2v[4];
        ld4_or_zero<T>(static_cast<const T*>(p.bias), ncol[b], nval[b], bv);
        ld4_or_zero<T>(static_cast<const T*>(p.bias2), ncol[b], nval[b], b2v);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[b][e] = bv[e] + b2v[e];
    }

    const int nq = p.cs / 64;
    // chunk qc's loads into buffer buf (LP + LB per wave, always)
    auto issue = [&](int qc, int buf) __attribute__((always_inline)) {
        const unsigned soff = static_cast<unsigned>(qc) * 128u;
        uint4* const base = &lds[buf * CHB * 64];
#pragma unroll
        for (int i = 0; i < LP; ++i) {
            const int b = wave + NW * i;        // wave-uniform
            const bool dead = HPBLK % NW != 0 && b >= HPBLK;
            if (NBUF == 1 && dead) break;
            buffer_load_lds(p.A, p.a_bytes, (lds_ptr_t)(base + (dead ? CHB - 1 : b) * 64), dead ? kOOB : voffP[i], soff);
        }
#pragma unroll
        for (int i = 0; i < LB; ++i) {
            const int b = wave + NW * i;
            const bool dead = NBB % NW != 0 && b >= NBB;
            if (NBUF == 1 && dead) break;
            buffer_load_lds(p.B, p.b_bytes, (lds_ptr_t)(base + (dead ? CHB - 1 : HPBLK + b) * 64), dead ? kOOB : voffB[i],
                            soff);
        }
    };
    static_assert(LP + LB <= 63, "the wait below counts the next chunk's loads");
    if constexpr (NBUF == 2) issue(0, 0);
    for (int qc = 0; qc < nq; ++qc) {
        if constexpr (NBUF == 2) {
            // the next chunk goes out before this one is waited for; its loads are the last issued
            if (qc + 1 < nq) {
                issue(qc + 1, (qc + 1) & 1);
                asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LP + LB) : "memory");
            } else {
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            }
        } else {
            if (qc > 0) __syncthreads();        // the previous chunk's fragments have been read
            issue(qc, 0);
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        }
        __builtin_amdgcn_s_barrier();           // every wave's share of chunk qc has landed
        const unsigned lds0 =
            static_cast<unsigned>(reinterpret_cast<size_t>((lds_ptr_t)(&lds[(NBUF == 2 ? qc & 1 : 0) * CHB * 64])));
#pragma unroll
        for (int tap = 0; tap < 9; ++tap) {
            const int pp = ((pix >> 3) + tap / 3) * PW + (pix & 7) + tap % 3;
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const int ch = 4 * ks + (lane >> 4);
                u32x4 af = lds_read16(lds0 + static_cast<unsigned>(pp * 128 + ((ch ^ (pp & 7)) << 4)));
                u32x4 bf[FN];
#pragma unroll
                for (int b = 0; b < FN; ++b) {
                    const int nb = b * 16 + (lane & 15);
                    bf[b] = lds_read16(lds0 + static_cast<unsigned>((HPBLK * 64 + (tap * BN + nb) * 8 + (ch ^ (nb & 7))) * 16));
                }
                lds_wait();
                pin(af);
#pragma unroll
                for (int b = 0; b < FN; ++b) {
                    pin(bf[b]);
                    acc[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, bf[b]),
                                                                   __builtin_bit_cast(bf16x8, af), acc[b], 0, 0, 0);
                }
            }
        }
        if constexpr (NBUF == 2) __syncthreads();   // chunk qc's buffer is read before chunk qc + 2 reuses it
    }

    if (!row_ok) return;
    const T* resp = static_cast<const T*>(p.res);
#pragma unroll
    for (int b = 0; b < FN; ++b) {
        if (nval[b] == 0) continue;
        const int64_t idx = row * p.ldc + ncol[b];
        float v[4], rv[4] = {0.f, 0.f, 0.f, 0.f};
        if (resp) ld4<T>(resp, idx, nval[b], rv);
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = act_f(acc[b][e] + rv[e], p.act);
        if (p.out_f32)
            store4<float>(static_cast<float*>(p.C), idx, v, nval[b]);
        else
            store4<T>(static_cast<T*>(p.C), idx, v, nval[b]);
    }
}

template <int BN, int TH, int NBUF>
static hipError_t launch_halo(const GemmParams& params, int width, hipStream_t st) {
    GemmParams p = params;
    const int64_t nt = (width + BN - 1) / BN;
    const int ty = (p.out_h + TH - 1) / TH, tx = (p.out_w + HTW - 1) / HTW;
    const int64_t imgs = p.M / (static_cast<int64_t>(p.out_h) * p.out_w);
    const int64_t total = imgs * ty * tx * p.ksub * nt;
    if (total >= (int64_t(1) << 31) / 8 || static_cast<int64_t>(ty) * tx * p.ksub * nt >= (int64_t(1) << 31))
        return hipErrorInvalidValue;
    p.g_total = static_cast<int>(total);
    p.g_per_xcd = static_cast<int>((total + 7) / 8);
    p.g_nt = static_cast<int>(nt);
    p.g_cols = static_cast<int>(nt * p.ksub);
    p.g_q = p.N / p.ksub;
    p.g_rr = p.N % p.ksub;
    p.g_div_group = FastDiv(static_cast<unsigned>(p.g_cols));
    p.g_div_nt = FastDiv(static_cast<unsigned>(nt));
    p.h_tiles = ty * tx;
    p.h_tx = tx;
    p.h_div_tiles = FastDiv(static_cast<unsigned>(ty * tx));
    p.h_div_tx = FastDiv(static_cast<unsigned>(tx));
    const int64_t grid = (total + 7) / 8 * 8;
    launch_kernel(conv3_halo_kernel<BN, TH, NBUF>, dim3(static_cast<unsigned>(grid)), dim3(TH * HTW / 16 * 64), 0, st,
                  p);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Tile selection.  All shapes share the K loop, so the choice only affects
// speed, never the bits of a result.
// ---------------------------------------------------------------------------

constexpr int kCUs = 256;

int gemm_splits(int64_t M, int N, int K, int dtype, int epi) {
    if (epi != EPI_STD || M * ((N + 3) / 4) >= (int64_t(1) << 31)) return 1;
    const int bk = dtype == MOPAR_BF16 ? 64 : 32;
    const int64_t nk = (K + bk - 1) / bk;
    const int64_t tiles = ((M + 63) / 64) * ((N + 63) / 64);   // reference tiling, independent of k
    // the reduce pass costs about as much as a dozen k stages: split only long K loops
    if (nk < 24) return 1;
    int s = 1;
    while (s < 16 && tiles * s < kCUs && nk / (2 * s) >= 4) s *= 2;
    return s;
}

template <typename T, int BM, int BN, int WM, int WN, int NS, int KH = 1, int KS = 1>
static hipError_t launch_cfg(const GemmParams& params, int width, hipStream_t st) {
    GemmParams p = params;
    const int64_t mt = (p.M + BM - 1) / BM, nt = (width + BN - 1) / BN;
    const int64_t total = mt * nt * p.ksub * p.splits;
    if (total >= (int64_t(1) << 31) / kGroupM) return hipErrorInvalidValue;
    p.g_mt = static_cast<int>(mt);
    p.g_nt = static_cast<int>(nt);
    p.g_total = static_cast<int>(total);
    p.g_per_xcd = static_cast<int>((total + 7) / 8);
    p.g_cols = static_cast<int>(nt * p.ksub * p.splits);
    p.g_nk = (p.K + 8 * Elt<T>::EPC - 1) / (8 * Elt<T>::EPC);
    p.g_q = p.N / p.ksub;
    p.g_rr = p.N % p.ksub;
    p.g_div_group = FastDiv(static_cast<unsigned>(kGroupM * p.g_cols));
    const int last = static_cast<int>(mt - (mt - 1) / kGroupM * kGroupM);   // m tiles in the last group
    p.g_div_last = FastDiv(static_cast<unsigned>(last));
    p.g_div_nt = FastDiv(static_cast<unsigned>(nt));
    p.g_div_ksub = FastDiv(static_cast<unsigned>(p.ksub));
    p.g_div_splits = FastDiv(static_cast<unsigned>(p.splits));
    if (p.conv) {
        const int bk = 8 * Elt<T>::EPC, dq = bk / p.cs;
        p.dc = bk - dq * p.cs;
        p.dqr = dq / p.kw;
        p.dqc = dq - p.dqr * p.kw;
        p.div_cs = FastDiv(static_cast<unsigned>(p.cs));
        p.div_kw = FastDiv(static_cast<unsigned>(p.kw));
    }
    const int64_t grid = (total + 7) / 8 * 8;
    const dim3 block(WM * WN * KS * 64);
    if (p.conv)
        launch_kernel((gemm_kernel<T, BM, BN, WM, WN, NS, KH, KS, true>), dim3(static_cast<unsigned>(grid)), block, 0,
                      st, p);
    else
        launch_kernel((gemm_kernel<T, BM, BN, WM, WN, NS, KH, KS, false>), dim3(static_cast<unsigned>(grid)), block, 0,
                      st, p);
    return hipGetLastError();
}

// 256 x 256 tiles (bf16, dense A, one split, standard epilogue)
static hipError_t launch_wide(const GemmParams& params, int width, hipStream_t st) {
    GemmParams p = params;
    p.c_bytes = static_cast<uint32_t>(((p.M - 1) * p.ldc + p.N) * (p.out_f32 ? 4 : 2));
    const int64_t mt = (p.M + 255) / 256, nt = (width + 255) / 256;
    const int64_t total = mt * nt * p.ksub;
    if (total >= (int64_t(1) << 31) / kWideGroupM) return hipErrorInvalidValue;
    p.g_mt = static_cast<int>(mt);
    p.g_nt = static_cast<int>(nt);
    p.g_total = static_cast<int>(total);
    p.g_per_xcd = static_cast<int>((total + 7) / 8);
    p.g_cols = static_cast<int>(nt * p.ksub);
    p.g_nk = (p.K + 63) / 64;
    p.g_q = p.N / p.ksub;
    p.g_rr = p.N % p.ksub;
    p.g_div_group = FastDiv(static_cast<unsigned>(kWideGroupM * p.g_cols));
    const int last = static_cast<int>(mt - (mt - 1) / kWideGroupM * kWideGroupM);
    p.g_div_last = FastDiv(static_cast<unsigned>(last));
    p.g_div_nt = FastDiv(static_cast<unsigned>(nt));
    if (p.wide_ctr && !p.res && p.act == MOPAR_ACT_NONE) {
        // persistent: one block per CU, tiles from per-XCD counters zeroed here
        if (p.g_nk < 2) return hipErrorInvalidValue;
        const hipError_t e = launch_fill_zero(p.wide_ctr, kWideCtrBytes, st);
        if (e != hipSuccess) return e;
        launch_kernel(gemm_wide_persistent, dim3(static_cast<unsigned>(kCUs)), dim3(256), 0, st, p);
        return hipGetLastError();
    }
    const int64_t grid = (total + 7) / 8 * 8;
    launch_kernel(gemm_wide_kernel<kWideBStages>, dim3(static_cast<unsigned>(grid)), dim3(256), 0, st, p);
    return hipGetLastError();
}

// Whether an operator runs on gemm_wide_kernel (and so on the 32 x 32 x 16 MFMA): dense bf16
// with the standard epilogue, not a boundary codec layer, K of at least 256, and at least four
// rounds of 256 x 256 tiles over the whole (M, N) -- with fewer, the block's unhidden set-up and
// epilogue cost more than its faster K loop saves (measured).  A function of the operator's
// (M, N, K) alone, never of the sub-slice count, so all its sub-slice launches take the same path.
static bool wide_class(const GemmParams& p) {
    // (the output span is addressed with 32-bit offsets, below the out-of-range offset 2^31)
    const int64_t c_span = ((p.M - 1) * p.ldc + p.N) * (p.out_f32 ? 4 : 2);
    return !p.conv && !p.thin && p.epi == EPI_STD && p.splits == 1 && p.K >= 256 && p.M >= 512 && p.N >= 512 &&
           ((p.M + 255) / 256) * ((p.N + 255) / 256) >= 4 * kCUs && c_span < (int64_t(1) << 31);
}

template <typename T>
static hipError_t dispatch(const GemmParams& p, hipStream_t st) {
    const int width = (p.N + p.ksub - 1) / p.ksub;   // widest sub-slice
    if constexpr (sizeof(T) == 2) {
        if (wide_class(p)) return launch_wide(p, width, st);
    }
    // few rows: the four waves split K (four 64-wide sub-stages per stage) instead of the tile
    if (p.M <= 16) return launch_cfg<T, 16, 64, 1, 1, 3, 4, 4>(p, width, st);
    // the LSTM step: 32 x 16 tiles (twice the blocks of 64 x 16, less LDS each) measured
    // fastest, alone and beside other streams' kernels
    if (p.epi == EPI_LSTM) return launch_cfg<T, 32, 16, 1, 1, 2, 4, 4>(p, width, st);
    if (p.M <= 64) {
        if (width >= 64) return launch_cfg<T, 64, 64, 1, 1, 2, 4, 4>(p, width, st);
        return launch_cfg<T, 64, 16, 1, 1, 3, 4, 4>(p, width, st);
    }
    const int64_t mt = (p.M + 127) / 128;
    auto blocks = [&](int64_t bm_tiles, int bn) { return bm_tiles * ((width + bn - 1) / bn) * p.ksub * p.splits; };
    // a codec layer with at most 128 output columns whose 64-row tiles would not give every
    // compute unit a block: 32 x 32 tiles (measured about 20 % faster on such encoders, cold)
    if (p.thin && width <= 128 && blocks((p.M + 63) / 64, width >= 64 ? 64 : 32) < kCUs)
        return launch_cfg<T, 32, 32, 2, 2, 4>(p, width, st);
    // 128-wide tiles unless they would leave more than a tenth of the columns they cover empty
    const bool w128 = width >= 128 && (width + 127) / 128 * 128 * 10 <= width * 11;
    if (w128 && blocks(mt, 128) >= kCUs) return launch_cfg<T, 128, 128, 2, 4, 2>(p, width, st);
    if (width >= 64 && blocks(mt, 64) >= kCUs) return launch_cfg<T, 128, 64, 4, 2, 3>(p, width, st);
    if (width >= 64) return launch_cfg<T, 64, 64, 2, 4, 4>(p, width, st);
    if (width >= 32) {
        if (blocks(mt, 32) >= kCUs) return launch_cfg<T, 128, 32, 4, 2, 3>(p, width, st);
        return launch_cfg<T, 64, 32, 4, 2, 4>(p, width, st);
    }
    // 16-column sub-slices: 64 x 16 tiles measured faster than 128 x 16 at every grid size tried
    return launch_cfg<T, 64, 16, 4, 1, 4>(p, width, st);
}

hipError_t launch_gemm(const GemmParams& params, int dtype, hipStream_t stream) {
    GemmParams p = params;
    if (p.splits < 1) p.splits = 1;
    if (p.ksub < 1) p.ksub = 1;
    if (p.conv) {
        p.div_hw = FastDiv(static_cast<unsigned>(p.out_h * p.out_w));
        p.div_w = FastDiv(static_cast<unsigned>(p.out_w));
    }
    if (p.M <= 0 || p.N <= 0) return hipSuccess;
    if (p.M > (int64_t(1) << 31) - 256) return hipErrorInvalidValue;   // rows are 32-bit in the kernel
    // operands are read through buffer resources with 32-bit byte offsets, and offset 2^31
    // must lie past both of them
    const int64_t esz = dtype == MOPAR_BF16 ? 2 : 4;
    const int64_t a_bytes = p.conv ? p.M / (int64_t(p.out_h) * p.out_w) * p.img_h * p.img_w * p.cs * esz
                                   : p.M * p.lda * esz;
    const int64_t b_bytes = int64_t(p.N) * p.K * esz;
    if (a_bytes >= (int64_t(1) << 31) || b_bytes >= (int64_t(1) << 31)) return hipErrorInvalidValue;
    p.a_bytes = static_cast<uint32_t>(a_bytes);
    p.b_bytes = static_cast<uint32_t>(b_bytes);
    // the reduce keeps every split's partial in flight at once, for at most 16 splits
    if (p.splits < 1 || p.splits > 16 || (p.splits > 1 && (!p.partial || p.epi != EPI_STD)))
        return hipErrorInvalidValue;
    if (p.conv && conv_halo_ok(dtype, p.kh, p.kw, p.stride, p.pad, p.cs, p.N, p.out_h, p.out_w, p.M)) {
        if (p.splits != 1 || p.epi != EPI_STD) return hipErrorInvalidValue;
        // 16-column tiles at every width (measured at least as fast as 32 on 32-wide sub-slices)
        const int width = (p.N + p.ksub - 1) / p.ksub;
        return p.cs / 64 > 2 ? launch_halo<16, 8, 2>(p, width, stream) : launch_halo<16, 8, 1>(p, width, stream);
    }
    hipError_t e = dtype == MOPAR_BF16 ? dispatch<__bf16>(p, stream) : dispatch<float>(p, stream);
    if (e != hipSuccess || p.splits == 1) return e;
    const int64_t n = p.M * ((p.N + 3) / 4);
    if (n >= (int64_t(1) << 31)) return hipErrorInvalidValue;
    p.r_div_groups = FastDiv(static_cast<unsigned>((p.N + 3) / 4));
    const unsigned blocks = static_cast<unsigned>((n + 255) / 256);
    if (dtype == MOPAR_BF16)
        launch_kernel(splitk_reduce_kernel<__bf16>, dim3(blocks), dim3(256), 0, stream, p);
    else
        launch_kernel(splitk_reduce_kernel<float>, dim3(blocks), dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace mopar
