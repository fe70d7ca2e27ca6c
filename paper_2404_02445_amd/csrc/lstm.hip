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
//   sequence and keeps its 64 x H slice of W_hh in registers (16 rows per wave, H / 32
//   16-byte MFMA fragments per lane).  Its four waves each run v_mfma_f32_16x16x32_bf16
//   with the weight fragment first, so a lane's four accumulators are gates i, f, g, o of
//   one (unit, batch row) pair and the cell update needs no exchange.
// * Steps.  Tiles of different 16-row batch groups never depend on each other; within a
//   group, step t needs every tile of step t - 1 (all of h_{t-1} for its rows).  A tile
//   stores its h_t and c_t with agent-coherent (sc1) 16-byte stores, waits until they have
//   completed, then marks its (step, tile) word done with one more coherent store.  A block
//   starting step t has one wave poll the group's words of step t - 1 (one lane per tile)
//   with agent-coherent loads, then reads h_{t-1} and c_{t-1} the same way.  No fence is
//   needed (the data moves only through coherent accesses), so no cache-wide write-back or
//   invalidate is issued, and no word is the target of every block's atomics.
// * Progress whatever the residency.  A tile is computed by whoever claims it (an atomic on
//   its (step, tile) word): a block claims all steps of its own tile when it starts.  A block
//   that has waited a while for a step claims that step's unclaimed tiles of its group and
//   computes them itself, reading the tile's W_hh rows from memory.  So blocks never wait for
//   a block that is not running: any one resident block finishes the whole sequence, and
//   several such kernels (other streams, other layers) sharing the GPU cannot hold each
//   other up.  A tile's result does not depend on which block computes it (same operands,
//   same MFMA order).
// * A poll limit far above any real wait ends the kernel with NaN in its tile's outputs
//   should progress ever stop, instead of letting it spin.
#include <cstdlib>

#include "internal.h"

namespace mopar {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCoherent = 16;          // buffer cache policy: agent scope (sc1)
constexpr int kRsrcWord3 = 0x00020000;
constexpr unsigned kOOB = 0x80000000u; // a buffer offset past every resource here: loads read zeros
constexpr int kGrace = 64;             // polls of a step counter before helping with that step
constexpr int kPollLimit = 1 << 22;    // polls without progress before giving up (~seconds)
constexpr int kDone = 1 << 24;         // added to a (step, tile) word once the tile's outputs are stored
constexpr int kMaxSteps = 4096;        // steps of one launch (the owner's claims are a bitmask in LDS)

struct LstmRecParams {
    const float* gx;      // [B * T][4H] gate pre-activations, biases included
    const __bf16* whh;    // [4H][H], row 4u + g = gate g (i, f, g, o) of unit u
    __bf16* hseq;         // [B][T][H] hidden states: the op's output, and h_{t-1} of step t
    float* cst;           // [B][H] cell state
    int* claim;           // [T][nb * ng] per (step, tile): 0 free, >= 1 claimed, >= kDone done
    int B, T, H, ng, nb;
    uint32_t h_bytes, c_bytes, w_bytes;
    int absent;           // test hook: > 1 makes blocks j with j % absent == 1 exit at once
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0), static_cast<int>(bytes),
                                             kRsrcWord3);
}

__device__ __forceinline__ int load_coherent(const int* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ float sigm(float v) { return 1.0f / (1.0f + __expf(-v)); }

template <int KF>
struct Tile {
    static constexpr int KP = KF * 32;            // K padded to whole MFMA steps
    static constexpr int RS = KP * 2 + 16;        // LDS row stride of the staged h rows (bytes)
};

// One tile (step t, gate slice jg of batch group jb): h_{t-1} rows into LDS, the product on
// MFMA (the owner's weights from registers, a helper's from memory), the cell, and the
// coherent stores of h_t and c_t.  Every thread of the block calls it.
template <int KF, bool OWNER>
__device__ __forceinline__ void compute_tile(const LstmRecParams& p, int t, int jg, int jb, const u32x4* wreg, float* creg,
                             bool cvalid, unsigned char* hs, float* oc, __bf16* oh) {
    constexpr int RS = Tile<KF>::RS, CPR = Tile<KF>::KP / 8;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int H = p.H, T = p.T, b0 = jb * 16;
    const auto hr = rsrc(p.hseq, p.h_bytes);
    const auto cr = rsrc(p.cst, p.c_bytes);
    const int bl = lane & 15, b = b0 + bl;
    const bool bok = b < p.B;
    const int g = jg * 64 + 16 * w + 4 * (lane >> 4);   // first of this lane's four gate rows
    const int u = g >> 2;
    const int G4 = 4 * H;
    // gate pre-activations (independent of the previous step: issued first)
    f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    if (bok) acc0 = *reinterpret_cast<const f32x4*>(p.gx + (static_cast<int64_t>(b) * T + t) * G4 + g);
    if (t > 0) {
        // h_{t-1} of the group's 16 rows: every load in flight at once (an offset past the
        // resource reads zeros: K padding and rows past B), then into LDS
        constexpr int NQ = (16 * CPR + 255) / 256;
        u32x4 v[NQ];
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int i = tid + 256 * q, r = i / CPR, c = i - r * CPR, bb = b0 + r;
            const bool ok = i < 16 * CPR && bb < p.B && 8 * c < H;
            const unsigned off = ok ? ((static_cast<uint32_t>(bb) * T + (t - 1)) * H + 8 * c) * 2 : kOOB;
            v[q] = __builtin_amdgcn_raw_buffer_load_b128(hr, static_cast<int>(off), 0, kCoherent);
        }
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int i = tid + 256 * q, r = i / CPR, c = i - r * CPR;
            if (i < 16 * CPR) *reinterpret_cast<u32x4*>(hs + r * RS + 16 * c) = v[q];
        }
    }
    float cprev = 0.0f;
    if (t > 0 && bok)
        cprev = cvalid ? *creg
                       : __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                       cr, static_cast<int>((b * H + u) * 4), 0, kCoherent));
    __syncthreads();
    f32x4 acc[4] = {acc0, acc1, acc1, acc1};
    if (t > 0) {
        // h fragments from LDS a batch at a time (their reads overlap), MFMAs spread over four
        // accumulators (fragment f into acc[f % 4], added in a fixed order below).  The owner's
        // weights are in registers (batches of four); a helper reads them from memory, two per
        // batch, so the helper path adds few registers to the owner's live weight slice.
        constexpr int NB = OWNER ? (KF < 4 ? KF : 4) : 2;
        const unsigned char* hrow = hs + bl * RS + 16 * (lane >> 4);
        const auto wr = rsrc(p.whh, p.w_bytes);
        const unsigned wbase = ((jg * 64 + 16 * w + bl) * H + 8 * (lane >> 4)) * 2;
#pragma unroll
        for (int f0 = 0; f0 < KF; f0 += NB) {
            u32x4 hv[NB], wv[NB];
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                hv[j] = *reinterpret_cast<const u32x4*>(hrow + 64 * (f0 + j));
                if constexpr (OWNER) {
                    wv[j] = wreg[f0 + j];
                } else {
                    const bool ok = 32 * (f0 + j) + 8 * (lane >> 4) < H;
                    wv[j] = __builtin_amdgcn_raw_buffer_load_b128(
                        wr, static_cast<int>(ok ? wbase + 64u * (f0 + j) : kOOB), 0, 0);
                }
            }
#pragma unroll
            for (int j = 0; j < NB; ++j)
                acc[(f0 + j) & 3] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    __builtin_bit_cast(bf16x8, wv[j]), __builtin_bit_cast(bf16x8, hv[j]), acc[(f0 + j) & 3], 0, 0, 0);
        }
    }
    const f32x4 v = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    const float c = sigm(v[1]) * cprev + sigm(v[0]) * tanhf(v[2]);
    const float h = sigm(v[3]) * tanhf(c);
    if (creg) *creg = c;
    // the tile's outputs, [16 batch rows][16 units], through LDS so the stores are whole 16-byte chunks
    const int ul = 4 * w + (lane >> 4);
    oc[bl * 16 + ul] = c;
    oh[bl * 16 + ul] = static_cast<__bf16>(h);
    __syncthreads();
    if (tid < 96) {
        const int q = tid < 64 ? tid : tid - 64;
        const int r = tid < 64 ? q >> 2 : q >> 1, part = tid < 64 ? q & 3 : q & 1;
        if (b0 + r < p.B) {
            if (tid < 64) {
                const u32x4 val = *reinterpret_cast<const u32x4*>(oc + r * 16 + 4 * part);
                __builtin_amdgcn_raw_buffer_store_b128(val, cr, static_cast<int>(((b0 + r) * H + jg * 16 + 4 * part) * 4),
                                                       0, kCoherent);
            } else {
                const u32x4 val = *reinterpret_cast<const u32x4*>(oh + r * 16 + 8 * part);
                __builtin_amdgcn_raw_buffer_store_b128(
                    val, hr, static_cast<int>(((static_cast<uint32_t>(b0 + r) * T + t) * H + jg * 16 + 8 * part) * 2), 0,
                    kCoherent);
            }
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this thread's coherent stores have completed
    __syncthreads();                                     // ... and every thread's
    // done (no block adds to a claimed word any more: helpers only claim words they saw free)
    if (tid == 0)
        __hip_atomic_store(p.claim + t * (p.nb * p.ng) + jb * p.ng + jg, kDone, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// NaN into the tile's h outputs of every step: the visible mark of a kernel that stopped making
// progress (never expected; see the poll limit).
__device__ void poison_tile(const LstmRecParams& p, int jg, int jb) {
    const auto hr = rsrc(p.hseq, p.h_bytes);
    for (int i = threadIdx.x; i < 16 * p.T * 16; i += 256) {
        const int r = i / (p.T * 16), rem = i - r * p.T * 16, t = rem >> 4, uu = rem & 15;
        if (jb * 16 + r < p.B)
            __builtin_amdgcn_raw_buffer_store_b16(static_cast<unsigned short>(0xFFFF), hr,
                                                  static_cast<int>(((static_cast<uint32_t>(jb * 16 + r) * p.T + t) * p.H +
                                                                    jg * 16 + uu) * 2),
                                                  0, kCoherent);
    }
}

// Wait until every tile of step s in batch group jb has completed.  After a grace period of
// polls the block claims any of that step's tiles nobody has claimed and computes it itself
// (weights from memory).  False if progress stopped for kPollLimit polls (the tile of slice jg
// is then marked with NaN).
template <int KF>
__device__ __forceinline__ bool await_step(const LstmRecParams& p, int s, int jb, int jg, unsigned char* hs, float* oc,
                                           __bf16* oh, int* bcast) {
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    int polls = 0;             // polls since the last progress made by this block
    bool helping = false;      // past the grace period: claim any free tile of the step
    int* cl = p.claim + s * (p.nb * p.ng) + jb * p.ng;
    for (;;) {
        // wave 0: one lane per tile of the group; ballots of done and of free tiles
        if (w == 0) {
            const int v = lane < p.ng ? load_coherent(cl + lane) : kDone;
            const unsigned long long not_done = __ballot(v < kDone);
            const unsigned long long free_ = __ballot(v == 0);
            int pick = -2;                                 // -2: step finished
            if (not_done) {
                pick = -1;
                if (lane == 0 && (helping || polls + 1 > kGrace)) {
                    unsigned long long m = free_;
                    while (m) {
                        const int j = __builtin_ctzll(m);
                        m &= m - 1;
                        if (__hip_atomic_fetch_add(cl + j, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
                            pick = j;
                            break;
                        }
                    }
                }
            }
            if (lane == 0) *bcast = pick;
        }
        __syncthreads();
        const int pick = *bcast;
        __syncthreads();
        if (pick == -2) return true;
        if (pick >= 0) {
            compute_tile<KF, false>(p, s, pick, jb, nullptr, nullptr, false, hs, oc, oh);
            polls = 0;
            helping = true;
            continue;
        }
        if (++polls > kGrace) helping = true;
        if (polls > kPollLimit) {
            poison_tile(p, jg, jb);
            return false;
        }
        __builtin_amdgcn_s_sleep(2);
    }
}

// (at least two waves per SIMD: at most 256 registers per lane, so that a GEMM block of another
// stream fits beside this block on the same CU)
template <int KF>
__global__ __launch_bounds__(256, 2) void lstm_recurrence_kernel(const LstmRecParams p) {
    __shared__ __attribute__((aligned(16))) unsigned char hs[16 * Tile<KF>::RS];
    __shared__ __attribute__((aligned(16))) float oc[16 * 16];
    __shared__ __attribute__((aligned(16))) __bf16 oh[16 * 16];
    __shared__ int bcast;
    __shared__ unsigned mine_bits[kMaxSteps / 32];
    const int own = blockIdx.x;
    if (p.absent > 1 && own % p.absent == 1) return;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int jb = own / p.ng, jg = own - jb * p.ng;
    const int ntile = p.nb * p.ng;
    (void)lane;

    // the owned slice of W_hh: wave w holds gate rows 64 jg + 16 w .. + 15, fragment f = k 32 f ..
    u32x4 wreg[KF];
    {
        const __bf16* wrow = p.whh + static_cast<int64_t>(jg * 64 + 16 * w + (lane & 15)) * p.H + 8 * (lane >> 4);
#pragma unroll
        for (int f = 0; f < KF; ++f) {
            wreg[f] = u32x4{0u, 0u, 0u, 0u};
            if (32 * f + 8 * (lane >> 4) < p.H) wreg[f] = *reinterpret_cast<const u32x4*>(wrow + 32 * f);
        }
    }
    float creg = 0.0f;
    bool cvalid = false;   // creg holds c of this tile's previous step (the owner computed it)

    // claim every step of the owned tile at once (steps a helper took already stay the helper's)
    for (int i = tid; i < kMaxSteps / 32; i += 256) mine_bits[i] = 0u;
    __syncthreads();
    for (int t = tid; t < p.T; t += 256)
        if (__hip_atomic_fetch_add(p.claim + t * ntile + own, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0)
            atomicOr(&mine_bits[t >> 5], 1u << (t & 31));
    __syncthreads();

    for (int t = 0; t < p.T; ++t) {
        const bool mine = (mine_bits[t >> 5] >> (t & 31)) & 1u;
        if (t > 0 && mine && !await_step<KF>(p, t - 1, jb, jg, hs, oc, oh, &bcast)) return;
        if (mine) {
            compute_tile<KF, true>(p, t, jg, jb, wreg, &creg, cvalid, hs, oc, oh);
            cvalid = true;
        } else {
            cvalid = false;
        }
    }
    // the last step too: a tile whose owner never ran is computed before the kernel ends
    (void)await_step<KF>(p, p.T - 1, jb, jg, hs, oc, oh, &bcast);
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
    // the step counters and claims start at zero on every launch
    hipError_t e = launch_fill_zero(sync, lstm_recurrence_sync_bytes(batch, steps, hidden), s);
    if (e != hipSuccess) return e;
    const int kf = (hidden + 31) / 32;
    if (kf <= 2)
        launch_rec<2>(p, s);
    else if (kf <= 4)
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
