// LSTM recurrence in one launch per layer (gfx950, bf16).
//
//   g_t = gx_t + W_hh h_{t-1}      (gx_t = W_ih x_t + b_ih + b_hh, precomputed in float32)
//   c_t = sig(f) c_{t-1} + sig(i) tanh(g),   h_t = sig(o) tanh(c_t),   h_{-1} = c_{-1} = 0
//
// The recurrence is T dependent steps of a (B x H) by (H x 4H) product.  Launching one
// kernel per step costs a launch and a cold start per step and re-streams W_hh every
// step.  Here one launch runs every step:
//
// * Tiles.  A tile is 64 gate rows (16 hidden units, all four gates of each: the rows of
//   W_hh are interleaved by unit) by 16 batch rows.  Block j owns tile j for the whole
//   sequence and keeps its 64 x H slice of W_hh in registers.  The contraction over k is
//   split across the four waves: wave w holds the tile's 64 rows for its quarter of k and
//   loads that quarter of h_{t-1} straight into MFMA operand registers.  Each wave runs
//   v_mfma_f32_16x16x32_bf16 with the weight fragment first, so an accumulator lane holds
//   gates i, f, g, o of one (unit, batch row) pair.  The four waves' partial sums meet in
//   LDS and are added in a fixed order; wave w then finishes units 4w .. 4w + 3 of the tile.
// * Steps.  Tiles of different 16-row batch groups never depend on each other; within a
//   group, step t needs all of h_{t-1} for its rows.  Before the launch every element of
//   hseq is set to 0xFFFF, a bf16 NaN pattern the kernel never stores (a NaN h is stored
//   as the canonical quiet NaN).  hseq is written once per element per launch, so an
//   element that no longer holds the fill is final.  A tile stores h_t with agent-coherent
//   (sc1) 16-byte stores and goes on at once.  Each wave of a block computing step t polls
//   one 16-byte chunk per tile its quarter of h_{t-1} covers, then loads the quarter (first
//   through the caches, then coherently while any lane still finds the fill).  The data is
//   its own ready signal: no flag is raised after the store completes, there is no flag to
//   poll, and no fence (no cache-wide write-back or invalidate) is issued.
// * Progress whatever the residency.  A tile is computed by whoever claims it (an atomic on
//   its (step, tile) word).  A block claims every step of its own tile when it starts, so
//   the steps it owns are a suffix of the sequence: a helper claims a step of a tile only
//   once the step before is complete everywhere in the group, which the owner, had it
//   started, would have reached only after its claims.  A block that has waited a while
//   for h_{t-1} walks the group's steps from the last one it has seen complete: for the
//   first step with chunks still missing it claims the missing tiles nobody has claimed and
//   computes them (weights from memory; the step's input is complete, having been seen).
//   A tile computed by a helper also leaves its cell state in memory, stored before its h
//   (so whoever has seen the h of that step reads the c), for the next step's computer.
//   Any one resident block thus finishes the whole sequence, and several such kernels
//   (other streams, other layers) sharing the GPU cannot hold each other up.  A tile's
//   result does not depend on which block computes it (same operands, same MFMA order,
//   same summation order).
// * A block waiting for h_{t-1} helps only after 500 us of the 100 MHz real-time clock: an
//   owner that is not yet resident is mostly held up by another kernel's blocks, and waiting
//   for it beats computing its tiles with weights from memory.  A helper that sees no
//   progress for 2 s ends with NaN in its tile's outputs
//   instead of spinning on (never expected); the NaN also releases every block waiting on
//   that tile.
#include <cstdlib>

#include "internal.h"

namespace mopar {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCoherent = 16;                // buffer cache policy: agent scope (sc1)
constexpr int kRsrcWord3 = 0x00020000;
constexpr unsigned kOOB = 0x80000000u;       // a buffer offset past every resource here: loads read zeros
constexpr unsigned kEmpty = 0xFFFFu;         // an h element not stored yet (the launcher's fill)
constexpr unsigned short kNaN = 0x7FC0;      // what a NaN h is stored as
constexpr unsigned short kPoison = 0x7FC1;   // h of a tile whose block stopped waiting (never expected)
constexpr uint64_t kGraceTicks = 50000;      // 500 us (100 MHz clock): waiting for h_{t-1} before helping
constexpr int kPollSleep = 1;                // s_sleep units (64 clocks) between two polls of h_{t-1}
constexpr uint64_t kScanTicks = 1000;        // 10 us of probing between two scans of a step while helping
constexpr uint64_t kGiveUpTicks = 200000000; // 2 s without progress: give up (never expected)
constexpr int kWaitVm0 = 0x0F70;             // s_waitcnt vmcnt(0) (expcnt and lgkmcnt left alone)
constexpr int kMaxSteps = 4096;              // steps of one launch (the owner's claims are a bitmask in LDS)

struct LstmRecParams {
    const float* gx;      // [B * T][4H] gate pre-activations, biases included
    const __bf16* whh;    // [4H][H], row 4u + g = gate g (i, f, g, o) of unit u
    __bf16* hseq;         // [B][T][H] hidden states: the op's output, and h_{t-1} of step t; 0xFFFF until stored
    float* cst;           // [B][H] cell state left by a helper for the tile's next step
    int* claim;           // [T][nb * ng] per (step, tile): 0 free, >= 1 claimed
    int B, T, H, ng, nb;
    uint32_t h_bytes, c_bytes, w_bytes;
    int absent;           // test hook: > 1 makes blocks j with j % absent == 1 exit at once
    int late_us;          // test hook: > 0 makes blocks of slices jg % 3 == 2 wait that long before claiming
};

struct Lds {
    f32x4 red[4][4][64];            // partial sums [wave][row tile][lane]
    float oc[16 * 16];              // a tile's c_t, [batch row][unit]
    unsigned short oh[16 * 16];     // a tile's h_t, [batch row][unit]
    unsigned long long missing[3];  // tiles of a step with chunks still unwritten (three in rotation)
    unsigned mine[kMaxSteps / 32];  // steps of the owned tile this block claimed
    int ok[4];                      // per wave: its quarter of h_{t-1} was complete
    int bcast;
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0), static_cast<int>(bytes),
                                             kRsrcWord3);
}

__device__ __forceinline__ int load_coherent(const int* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The cell's nonlinearities from the hardware exponential and reciprocal (about 1 ulp each):
// sig(v) = 1 / (1 + e^-v), tanh(v) = 2 sig(2v) - 1.  Near v = 0 the tanh form loses relative
// (not absolute) precision, about 1e-7 absolute, far below the bf16 rounding of h.
// Every expression of the cell is written out operation by operation (contraction off): a tile
// computed by its owner and by a helper, inlined in different contexts, must round alike.
__device__ __forceinline__ float sigm(float v) {
#pragma clang fp contract(off)
    return __builtin_amdgcn_rcpf(1.0f + __expf(-v));
}
__device__ __forceinline__ float tanh_fast(float v) {
#pragma clang fp contract(off)
    return 2.0f * sigm(2.0f * v) - 1.0f;
}

__device__ __forceinline__ bool has_empty(u32x4 x) {
    bool e = false;
#pragma unroll
    for (int i = 0; i < 4; ++i) e |= (x[i] & 0xFFFFu) == kEmpty || (x[i] >> 16) == kEmpty;
    return e;
}

// byte offset of the 16-byte chunk of h_{t-1} a lane feeds to fragment f (8 elements of row b)
__device__ __forceinline__ unsigned h_off(const LstmRecParams& p, int b, int t, int k) {
    return ((static_cast<uint32_t>(b) * p.T + t) * p.H + k) * 2;
}

__device__ __forceinline__ uint64_t now_ticks() { return __builtin_amdgcn_s_memrealtime(); }

// Wait (until the clock passes `deadline`) until the h of step f of the tiles whose units this wave's
// quarter of k covers appears written, judged by one 16-byte chunk per tile (the last row's
// second half): lane l polls tile 2 w KW + l.  Cheap (one load per tile) compared with the
// quarter itself, so a waiting wave does not flood memory; the quarter is checked in full
// afterwards.
template <int KW>
__device__ __forceinline__ void probe_quarter(const LstmRecParams& p, int f, int jb, uint64_t deadline) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int pt = 2 * w * KW + lane, b0 = jb * 16;
    const int rl = (p.B - b0 < 16 ? p.B - b0 : 16) - 1;
    const unsigned off = lane < 2 * KW && 16 * pt < p.H ? h_off(p, b0 + rl, f, 16 * pt + 8) : kOOB;
    const auto hr = rsrc(p.hseq, p.h_bytes);
    while (__ballot(has_empty(__builtin_amdgcn_raw_buffer_load_b128(hr, static_cast<int>(off), 0, kCoherent))) != 0 &&
           now_ticks() < deadline) {
    }
}

// The cell and the stores of one tile, after the gate pre-activations are known (v: gates
// i, f, g, o of this lane's (unit, batch row)).  A helper also stores c_t, completed before
// any h_t store is issued.
template <bool HELPER>
__device__ __forceinline__ void finish_tile(const LstmRecParams& p, int t, int jg, int jb, f32x4 v, float cprev,
                                            float* creg, Lds& s) {
#pragma clang fp contract(off)
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, bl = lane & 15, ul = 4 * w + (lane >> 4);
    const int b0 = jb * 16;
    const float c = __builtin_fmaf(sigm(v[1]), cprev, sigm(v[0]) * tanh_fast(v[2]));
    const float h = sigm(v[3]) * tanh_fast(c);
    if (creg) *creg = c;
    unsigned short hb = __builtin_bit_cast(unsigned short, static_cast<__bf16>(h));
    if ((hb & 0x7FFFu) > 0x7F80u) hb = kNaN;   // any NaN, whatever its payload
    s.oh[bl * 16 + ul] = hb;
    if (HELPER) s.oc[bl * 16 + ul] = c;
    __syncthreads();
    if (HELPER && t + 1 < p.T) {
        if (tid < 64) {
            const int r = tid >> 2, part = tid & 3;
            if (b0 + r < p.B)
                __builtin_amdgcn_raw_buffer_store_b128(*reinterpret_cast<const u32x4*>(s.oc + r * 16 + 4 * part),
                                                       rsrc(p.cst, p.c_bytes),
                                                       static_cast<int>(((b0 + r) * p.H + jg * 16 + 4 * part) * 4), 0,
                                                       kCoherent);
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this thread's c stores have completed
        __syncthreads();                                     // ... and every thread's
    }
    if (tid < 32) {
        const int r = tid >> 1, part = tid & 1;
        if (b0 + r < p.B) {
            const u32x4 val = *reinterpret_cast<const u32x4*>(s.oh + r * 16 + 8 * part);
            __builtin_amdgcn_raw_buffer_store_b128(val, rsrc(p.hseq, p.h_bytes),
                                                   static_cast<int>(h_off(p, b0 + r, t, jg * 16 + 8 * part)), 0,
                                                   kCoherent);
        }
    }
}

// Partial sums of the four waves added in a fixed order, plus the input projection.
__device__ __forceinline__ f32x4 reduce_gates(const Lds& s, f32x4 gxv) {
#pragma clang fp contract(off)
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    return gxv + ((s.red[0][w][lane] + s.red[1][w][lane]) + (s.red[2][w][lane] + s.red[3][w][lane]));
}

__device__ __forceinline__ f32x4 load_gx(const LstmRecParams& p, int t, int jg, int jb) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int b = jb * 16 + (lane & 15), u = jg * 16 + 4 * w + (lane >> 4);
    f32x4 g = {0.f, 0.f, 0.f, 0.f};
    if (b < p.B) g = *reinterpret_cast<const f32x4*>(p.gx + (static_cast<int64_t>(b) * p.T + t) * (4 * p.H) + 4 * u);
    return g;
}

__device__ __forceinline__ float load_c(const LstmRecParams& p, int jg, int jb) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int b = jb * 16 + (lane & 15), u = jg * 16 + 4 * w + (lane >> 4);
    if (b >= p.B) return 0.0f;
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rsrc(p.cst, p.c_bytes),
                                                                          static_cast<int>((b * p.H + u) * 4), 0,
                                                                          kCoherent));
}

// The owner's step t of its tile.  False if some wave still found the fill in its quarter of
// h_{t-1} after the grace period (nothing is stored then).
template <int KF>
__device__ __forceinline__ bool own_step(const LstmRecParams& p, int t, int jg, int jb, const u32x4* wreg, float& creg,
                                         bool cvalid, Lds& s) {
    constexpr int KW = KF / 4;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, kg = lane >> 4;
    const int b = jb * 16 + (lane & 15);
    f32x4 v = load_gx(p, t, jg, jb);
    if (t == 0) {
        finish_tile<false>(p, t, jg, jb, v, 0.0f, &creg, s);
        return true;
    }
    const auto hr = rsrc(p.hseq, p.h_bytes);
    const int k0 = 32 * w * KW + 8 * kg;
    const unsigned base = b < p.B ? h_off(p, b, t - 1, k0) : kOOB;
    const uint64_t deadline = now_ticks() + kGraceTicks;
    u32x4 hv[KW];
    bool wave_ok = false;
    // wait until one chunk of every tile of the wave's quarter shows data (a cheap probe, so
    // that waiting waves do not flood memory with full loads), then load the quarter: first
    // through the caches, so that the tiles of the group running on one XCD can share one
    // fetch of a line through its L2 (a cached copy can only be older than memory, and an
    // element that differs from the fill is final), then, while any lane still finds the
    // fill, again as a whole with coherent loads
    probe_quarter<KW>(p, t - 1, jb, deadline);
    {
        bool e = false;
#pragma unroll
        for (int j = 0; j < KW; ++j) {
            hv[j] = __builtin_amdgcn_raw_buffer_load_b128(
                hr, static_cast<int>(base != kOOB && k0 + 32 * j < p.H ? base + 64 * j : kOOB), 0, 0);
            e |= has_empty(hv[j]);
        }
        wave_ok = __ballot(e) == 0;
    }
    while (!wave_ok && now_ticks() < deadline) {
        __builtin_amdgcn_s_sleep(kPollSleep);
        bool e = false;
#pragma unroll
        for (int j = 0; j < KW; ++j) {
            hv[j] = __builtin_amdgcn_raw_buffer_load_b128(
                hr, static_cast<int>(base != kOOB && k0 + 32 * j < p.H ? base + 64 * j : kOOB), 0, kCoherent);
            e |= has_empty(hv[j]);
        }
        wave_ok = __ballot(e) == 0;
    }
    // (run whatever the poll's outcome: the sums of an incomplete h_{t-1} are discarded)
    f32x4 acc[4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < KW; ++j)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
            acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wreg[mt * KW + j]),
                                                              __builtin_bit_cast(bf16x8, hv[j]), acc[mt], 0, 0, 0);
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) s.red[w][mt][lane] = acc[mt];
    if (lane == 0) s.ok[w] = wave_ok;
    __syncthreads();
    if (!(s.ok[0] && s.ok[1] && s.ok[2] && s.ok[3])) {
        __syncthreads();   // every wave has read the flags before anything reuses them
        return false;
    }
    v = reduce_gates(s, v);
    // c_{t-1}: the owner's own from the last step, else (its first step) the helper's, whose
    // store completed before its h_{t-1}, which this block has now seen.  (The load is waited
    // for inside the branch: no wait for it is left on the common path.)
    float cprev = creg;
    if (!cvalid) {
        cprev = load_c(p, jg, jb);
        asm volatile("" : "+v"(cprev));
    }
    finish_tile<false>(p, t, jg, jb, v, cprev, &creg, s);
    return true;
}

// A helper's step t of tile (jg, jb), h_{t-1} of the group already seen complete: weights
// from memory, the same operands, MFMA order and summation order as the owner's.
template <int KF>
__device__ void help_step(const LstmRecParams& p, int t, int jg, int jb, Lds& s) {
    constexpr int KW = KF / 4;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, kg = lane >> 4;
    const int b = jb * 16 + (lane & 15);
    f32x4 v = load_gx(p, t, jg, jb);
    float cprev = 0.0f;
    if (t > 0) {
        const auto hr = rsrc(p.hseq, p.h_bytes);
        const auto wr = rsrc(p.whh, p.w_bytes);
        f32x4 acc[4];
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
        for (int j = 0; j < KW; ++j) {
            const int k = 32 * (w * KW + j) + 8 * kg;
            const u32x4 hv = __builtin_amdgcn_raw_buffer_load_b128(
                hr, static_cast<int>(b < p.B && k < p.H ? h_off(p, b, t - 1, k) : kOOB), 0, kCoherent);
            u32x4 wv[4];
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
                wv[mt] = __builtin_amdgcn_raw_buffer_load_b128(
                    wr, static_cast<int>(k < p.H ? ((jg * 64 + 16 * mt + (lane & 15)) * p.H + k) * 2 : kOOB), 0, 0);
#pragma unroll
            for (int mt = 0; mt < 4; ++mt)
                acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wv[mt]),
                                                                  __builtin_bit_cast(bf16x8, hv), acc[mt], 0, 0, 0);
        }
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) s.red[w][mt][lane] = acc[mt];
        cprev = load_c(p, jg, jb);
        __syncthreads();
        v = reduce_gates(s, v);
    }
    finish_tile<true>(p, t, jg, jb, v, cprev, nullptr, s);
    __syncthreads();   // the staged outputs have been read before the next tile reuses them
}

// Make steps up to `target` complete in batch group jb.  v is the last step this block has
// seen complete in the group (-1: none); it walks on from there.  At the first step with
// chunks still unwritten it claims one of the tiles involved that nobody has claimed and
// computes it; if all are claimed it waits for them.  `it` counts iterations across calls (the
// three missing-tile masks rotate with it).  False if no progress was seen for kGiveUpTicks
// (thread 0's clock decides, so the block leaves together).
template <int KF>
__device__ bool help_until(const LstmRecParams& p, int target, int jb, int& v, int& it, Lds& s) {
    const int tid = threadIdx.x, CH = p.H / 8, ntile = p.nb * p.ng;
    const auto hr = rsrc(p.hseq, p.h_bytes);
    uint64_t last = now_ticks();   // last progress (used by thread 0)
    for (; v < target; ++it) {
        const int f = v + 1;
        unsigned long long miss = 0;
        for (int i = tid; i < 16 * CH; i += 256) {
            const int r = i / CH, c = i - r * CH, b = jb * 16 + r;
            if (b < p.B && has_empty(__builtin_amdgcn_raw_buffer_load_b128(hr, static_cast<int>(h_off(p, b, f, 8 * c)),
                                                                           0, kCoherent)))
                miss |= 1ull << (c >> 1);
        }
        // the mask used two iterations ago is cleared for the next one (read by everyone
        // before the last barrier, first written after the next)
        if (tid == 0) s.missing[(it + 1) % 3] = 0ull;
        if (miss) atomicOr(&s.missing[it % 3], miss);
        __syncthreads();
        const unsigned long long m = s.missing[it % 3];
        if (m == 0) {
            v = f;
            last = now_ticks();
            continue;
        }
        if (tid == 0) {
            int pick = -1;
            for (unsigned long long r = m; r != 0 && pick < 0; r &= r - 1) {
                const int j = __builtin_ctzll(r);
                int* cw = p.claim + f * ntile + jb * p.ng + j;
                if (load_coherent(cw) == 0 &&
                    __hip_atomic_fetch_add(cw, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0)
                    pick = j;
            }
            if (pick < 0 && now_ticks() - last > kGiveUpTicks) pick = -2;
            s.bcast = pick;
        }
        __syncthreads();
        const int pick = s.bcast;
        if (pick == -2) return false;
        if (pick >= 0) {
            help_step<KF>(p, f, pick, jb, s);
            last = now_ticks();
        } else {
            probe_quarter<KF / 4>(p, f, jb, now_ticks() + kScanTicks);   // no flood of scans while waiting
        }
    }
    return true;
}

// NaN into the tile's h outputs of every step: the visible mark of a kernel that stopped making
// progress (never expected; see kGiveUpTicks).  Being unlike the fill, it also releases blocks
// waiting on the tile.
__device__ void poison_tile(const LstmRecParams& p, int jg, int jb) {
    const auto hr = rsrc(p.hseq, p.h_bytes);
    for (int i = threadIdx.x; i < 16 * p.T * 16; i += 256) {
        const int r = i / (p.T * 16), rem = i - r * p.T * 16, t = rem >> 4, uu = rem & 15;
        if (jb * 16 + r < p.B)
            __builtin_amdgcn_raw_buffer_store_b16(kPoison, hr, static_cast<int>(h_off(p, jb * 16 + r, t, jg * 16 + uu)), 0,
                                                  kCoherent);
    }
}

// (at least two waves per SIMD: at most 256 registers per lane, so that a GEMM block of another
// stream fits beside this block on the same CU)
template <int KF>
__global__ __launch_bounds__(256, 2) void lstm_recurrence_kernel(const LstmRecParams p) {
    constexpr int KW = KF / 4;
    __shared__ Lds s;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int own = blockIdx.x;
    const int jb = own / p.ng, jg = own - jb * p.ng;
    if (p.absent > 1 && jg % p.absent == 1) return;
    const int ntile = p.nb * p.ng;

    // the owned slice of W_hh: wave w holds gate rows 64 jg + 16 mt + (lane & 15) of row tile mt,
    // fragment j = k 32 (w KW + j) + 8 (lane >> 4) .. + 7
    u32x4 wreg[4 * KW];
    {
        const auto wr = rsrc(p.whh, p.w_bytes);
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int j = 0; j < KW; ++j) {
                const int k = 32 * (w * KW + j) + 8 * (lane >> 4);   // past H: reads zeros
                wreg[mt * KW + j] = __builtin_amdgcn_raw_buffer_load_b128(
                    wr, static_cast<int>(k < p.H ? ((jg * 64 + 16 * mt + (lane & 15)) * p.H + k) * 2 : kOOB), 0, 0);
            }
    }

    // (the weight loads complete here: no wait for them is placed inside the step loop, where
    // it would also wait for the wave's latest h store, the counter retiring in issue order)
    __builtin_amdgcn_s_waitcnt(kWaitVm0);

    if (p.late_us > 0 && jg % 3 == 2) {   // test hook: an owner that starts late
        const uint64_t until = now_ticks() + 100ull * static_cast<uint64_t>(p.late_us);
        while (now_ticks() < until) __builtin_amdgcn_s_sleep(8);
    }

    // claim every step of the owned tile at once (steps a helper took already stay the helper's)
    for (int i = tid; i < kMaxSteps / 32; i += 256) s.mine[i] = 0u;
    if (tid < 3) s.missing[tid] = 0ull;
    __syncthreads();
    for (int t = tid; t < p.T; t += 256)
        if (__hip_atomic_fetch_add(p.claim + t * ntile + own, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0)
            atomicOr(&s.mine[t >> 5], 1u << (t & 31));
    __syncthreads();

    int v = -1, it = 0;
    float creg = 0.0f;
    bool cvalid = false;   // creg holds c of this tile's previous step (this block computed it)
    for (int t = 0; t < p.T; ++t) {
        if (!((s.mine[t >> 5] >> (t & 31)) & 1u)) {
            cvalid = false;
            continue;
        }
        // (a step whose input this block has seen complete cannot fail again: the retry bound
        // only guards against looping forever should that ever not hold)
        for (int tries = 0; !own_step<KF>(p, t, jg, jb, wreg, creg, cvalid, s); ++tries) {
            if (tries == 2 || !help_until<KF>(p, t - 1, jb, v, it, s)) {
                poison_tile(p, jg, jb);
                return;
            }
        }
        if (v < t - 1) v = t - 1;
        cvalid = true;
    }
    // the last step too: a tile whose owner never ran is computed before the kernel ends
    if (!help_until<KF>(p, p.T - 1, jb, v, it, s)) poison_tile(p, jg, jb);
}

template <int KF>
void launch_rec(const LstmRecParams& p, hipStream_t s) {
    launch_kernel(lstm_recurrence_kernel<KF>, dim3(static_cast<unsigned>(p.ng * p.nb)), dim3(256), 0, s, p);
}

}  // namespace

bool lstm_recurrence_ok(int dtype, int64_t batch, int64_t steps, int64_t hidden) {
    return dtype == MOPAR_BF16 && hidden % 16 == 0 && hidden <= 1024 && steps <= kMaxSteps &&
           batch * steps * hidden * 2 < (int64_t(1) << 31) && batch * hidden * 4 < (int64_t(1) << 31);
}

size_t lstm_recurrence_sync_bytes(int64_t batch, int64_t steps, int64_t hidden) {
    const int64_t nb = (batch + 15) / 16, ng = hidden / 16;
    return static_cast<size_t>(steps * nb * ng) * sizeof(int);
}

hipError_t launch_lstm_recurrence(const float* gx, const void* whh, void* hseq, float* cst, void* sync, int batch,
                                  int steps, int hidden, hipStream_t s) {
    if (!lstm_recurrence_ok(MOPAR_BF16, batch, steps, hidden) || batch < 1 || steps < 1) return hipErrorInvalidValue;
    LstmRecParams p{};
    p.gx = gx;
    p.whh = static_cast<const __bf16*>(whh);
    p.hseq = static_cast<__bf16*>(hseq);
    p.cst = cst;
    p.B = batch;
    p.T = steps;
    p.H = hidden;
    p.ng = hidden / 16;
    p.nb = (batch + 15) / 16;
    p.claim = static_cast<int*>(sync);
    p.h_bytes = static_cast<uint32_t>(static_cast<int64_t>(batch) * steps * hidden * 2);
    p.c_bytes = static_cast<uint32_t>(static_cast<int64_t>(batch) * hidden * 4);
    p.w_bytes = static_cast<uint32_t>(int64_t(4) * hidden * hidden * 2);
    // test hook: simulate blocks that are never resident (their tiles must be computed by others)
    if (const char* e = getenv("MOPAR_TEST_LSTM_ABSENT")) p.absent = atoi(e);
    if (p.absent > 1 && p.ng < 2) p.absent = 0;
    if (const char* e = getenv("MOPAR_TEST_LSTM_LATE_US")) p.late_us = atoi(e);
    // claims start at zero and every h element at the fill on every launch
    hipError_t e = launch_fill_zero(sync, lstm_recurrence_sync_bytes(batch, steps, hidden), s);
    if (e == hipSuccess) e = launch_fill_bytes(hseq, p.h_bytes, 0xFF, s);
    if (e != hipSuccess) return e;
    const int kf = (hidden + 31) / 32;
    if (kf <= 4)
        launch_rec<4>(p, s);
    else if (kf <= 8)
        launch_rec<8>(p, s);
    else if (kf <= 16)
        launch_rec<16>(p, s);
    else
        launch_rec<32>(p, s);
    return hipGetLastError();
}

}  // namespace mopar
