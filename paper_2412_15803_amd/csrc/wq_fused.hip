// Decode linears with the elementwise work of a layer fused in (batch 1), and
// the argmax of the final logits.  The graph-level fusion the paper's compiler
// performs (Sec. 2.3), written by hand for the Llama-class decoders of
// Table 1: an RMSNorm or SiLU-gated prologue on x, a residual added to y
// before its single rounding.
//
// fused_m1_kernel<LPR, GPL> is the batch-1 GEMV of wq_kernels.hip (same row
// steps, buffer loads and two-buffer pipeline) with two changes:
//   * prologue: the block's 256 threads first compute x_eff for the whole row
//     into LDS, one round trip for x and the second operand (norm weight or
//     up half), a fixed-order block sum for RMSNorm, then one fp16 rounding
//     per element; each wave then stages its lanes' x_eff from LDS;
//   * epilogue: row sums are staged in LDS as fp32, and the residual is added
//     when y is written, so y is rounded once.
// argmax_kernel: one 1024-thread workgroup loads all logits in one round trip
// and reduces (value, index) pairs, the smaller index winning ties.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <cstdarg>
#include <cstdio>
#include <vector>

#include "wq_device.h"
#include "wq_fused.h"
#include "wq_internal.h"
#include "wq_plan.h"

namespace wq {
namespace fused {
namespace {

using namespace dev;

constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / kWave;
// Launch shape and loads, as for the single-linear GEMV: about 1024 waves,
// steps of four 16-byte loads per lane and non-temporal weight loads.
// Measured on the dependent 3B step (113 launches per token): 899 us per
// token with 2048 waves, six-load steps and the default policy; 857 with the
// loads past a wave's last step no longer reading the next wave's rows; 767
// with 1024 waves; 723 with four-load steps; 675-683 with non-temporal
// loads (512 waves: 870, 768: 740; two- or three-load steps: the same).
#ifndef WQ_FUSED_WAVES
#define WQ_FUSED_WAVES (256 * 4)
#endif
#ifndef WQ_FUSED_STEP_LOADS
#define WQ_FUSED_STEP_LOADS 4
#endif
#ifndef WQ_FUSED_CPOL
#define WQ_FUSED_CPOL kCpolNonTemporal
#endif
constexpr int kTargetWaves = WQ_FUSED_WAVES;
constexpr int kFLoads = WQ_FUSED_STEP_LOADS;
constexpr int kMaxK = (int)WQ_FUSED_MAX_K;
constexpr int kArgThreads = 1024;

struct Args {
    const u32x4* packed;
    const uint16_t* scales;
    const uint16_t* x;
    uint16_t* y;
    const uint16_t* norm;
    const uint16_t* residual;
    int64_t n;
    int64_t rows_per_wave;
    int ng;
    int prologue;
    float eps;
};

__device__ __forceinline__ float h2f(uint32_t bits16) { return __half2float(__ushort_as_half((uint16_t)bits16)); }
__device__ __forceinline__ uint32_t f2h(float v) { return __half_as_ushort(__float2half_rn(v)); }

// silu(a) = a / (1 + e^-a) with the hardware exp2 and reciprocal (about one
// ulp each): every block evaluates it for the whole row, and its fp32 error
// stays far below the fp16 rounding that follows.  Large negative a gives
// exp2 = inf and a * 0 = -0; large positive a gives exactly a.
__device__ __forceinline__ float silu(float a) {
    return a * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(a * -1.4426950408889634f));
}

// Sum over the block in a fixed order (every thread gets the same value).
__device__ __forceinline__ float block_sum(float v, float* red) {
    v = segment_sum<kWave>(v);  // the wave's total lands in its last lane
    if ((threadIdx.x & (kWave - 1)) == kWave - 1) red[threadIdx.x / kWave] = v;
    __syncthreads();
    float t = red[0];
#pragma unroll
    for (int w = 1; w < kWavesPerBlock; ++w) t += red[w];
    return t;
}

// x_eff of the whole row into LDS (all threads of the block take part): one
// round trip for x and the second operand (norm weight or up half), then
// `between()` (loads the caller wants in flight behind these), then the
// arithmetic, the LDS writes and a barrier.  CPT 8-element chunks of x per
// thread cover rows of up to 256 CPT groups.
template <int CPT, typename F>
__device__ __forceinline__ void stage_prologue(const Args& a, uint16_t* s_x, float* red, F between) {
    const int tid = threadIdx.x;
    const int chunks = a.ng * (kGroup / 8);
    const WQ_GLOBAL u32x4* xs = gbl(reinterpret_cast<const u32x4*>(a.x));
    const WQ_GLOBAL u32x4* bs = a.prologue == WQ_PROLOGUE_RMSNORM
                                    ? gbl(reinterpret_cast<const u32x4*>(a.norm))
                                    : gbl(reinterpret_cast<const u32x4*>(a.x)) + chunks;  // the up half
    u32x4 xa[CPT], xb[CPT];
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
        const int c = tid + r * kBlock;
        if (c < chunks) {
            xa[r] = xs[c];
            xb[r] = bs[c];
        }
    }
    load_order_fence();
    between();
    float inv = 0.0f;
    if (a.prologue == WQ_PROLOGUE_RMSNORM) {
        float ss = 0.0f;
#pragma unroll
        for (int r = 0; r < CPT; ++r) {
            if (tid + r * kBlock >= chunks) continue;
            const uint32_t w[4] = {xa[r].x, xa[r].y, xa[r].z, xa[r].w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float lo = h2f(w[i] & 0xFFFFu), hi = h2f(w[i] >> 16);
                ss = fmaf(lo, lo, ss);
                ss = fmaf(hi, hi, ss);
            }
        }
        const float total = block_sum(ss, red);
        inv = 1.0f / sqrtf(total / (float)(a.ng * kGroup) + a.eps);
    }
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
        const int c = tid + r * kBlock;
        if (c >= chunks) continue;
        const uint32_t wa[4] = {xa[r].x, xa[r].y, xa[r].z, xa[r].w};
        const uint32_t wb[4] = {xb[r].x, xb[r].y, xb[r].z, xb[r].w};
        uint32_t o[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float v[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const float p = h2f(h ? wa[i] >> 16 : wa[i] & 0xFFFFu);
                const float q = h2f(h ? wb[i] >> 16 : wb[i] & 0xFFFFu);
                v[h] = a.prologue == WQ_PROLOGUE_RMSNORM ? (p * inv) * q : silu(p) * q;
            }
            o[i] = f2h(v[0]) | (f2h(v[1]) << 16);
        }
        reinterpret_cast<u32x4*>(s_x)[c] = u32x4{o[0], o[1], o[2], o[3]};
    }
    __syncthreads();
}

// load_x_lane with x_eff already in LDS.
template <int LPR, int GPL>
__device__ __forceinline__ void load_x_lane_lds(const uint16_t* s_x, int ng, int lane, half2v (&xr)[GPL][16]) {
    const int sub = lane & (LPR - 1);
#pragma unroll
    for (int j = 0; j < GPL; ++j) {
        const bool act = sub + LPR * j < ng;
        const u32x4* src = reinterpret_cast<const u32x4*>(s_x + min(sub + LPR * j, ng - 1) * kGroup);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const u32x4 d = src[c];
            xr[j][4 * c + 0] = as_h2(act ? (d.x & 0xFFFFu) | (d.z << 16) : 0u);
            xr[j][4 * c + 1] = as_h2(act ? (d.x >> 16) | (d.z & 0xFFFF0000u) : 0u);
            xr[j][4 * c + 2] = as_h2(act ? (d.y & 0xFFFFu) | (d.w << 16) : 0u);
            xr[j][4 * c + 3] = as_h2(act ? (d.y >> 16) | (d.w & 0xFFFF0000u) : 0u);
        }
    }
}

// compute_step with the row sums staged as fp32 (the residual is added later).
template <int LPR, int GPL, int LOADS = WQ_STEP_LOADS>
__device__ __forceinline__ void compute_step_f32(const StepBuf& b, const half2v (&xr)[GPL][16], int nrows,
                                                 float* ylds, int yrel, int lane) {
    using S = StepShape<LPR, GPL, LOADS>;
    const int slot = lane / LPR;
    const int sub = lane & (LPR - 1);
#pragma unroll
    for (int u = 0; u < S::U; ++u) {
        float acc = 0.0f;
#pragma unroll
        for (int j = 0; j < GPL; ++j) {
            const float s = h2f(b.s[u * GPL + j]);
            acc = fmaf(s, dot_group(b.w[u * GPL + j], xr[j]), acc);
        }
        const float tot = segment_sum<LPR>(acc);
        const int rr = slot * S::U + u;
        if (sub == LPR - 1 && rr < nrows) ylds[yrel + rr] = tot;
    }
}

__device__ __forceinline__ void flush_y_residual(uint16_t* y, const uint16_t* residual, int64_t row0,
                                                 const float* ylds, int count, int lane) {
    wave_lds_sync();
    WQ_GLOBAL uint16_t* dst = gbl(y) + row0;
    if (residual) {
        const WQ_GLOBAL uint16_t* res = gbl(residual) + row0;
        for (int i = lane; i < count; i += kWave) dst[i] = (uint16_t)f2h(ylds[i] + h2f(res[i]));
    } else {
        for (int i = lane; i < count; i += kWave) dst[i] = (uint16_t)f2h(ylds[i]);
    }
    wave_lds_sync();
}

template <int LPR, int GPL>
__global__ __launch_bounds__(kBlock) void fused_m1_kernel(const Args a) {
    constexpr int R = StepShape<LPR, GPL, kFLoads>::ROWS;
    extern __shared__ __align__(16) uint16_t s_x[];  // x_eff, K entries (prologues only)
    __shared__ __align__(16) float s_y[kWavesPerBlock][kYRows];
    __shared__ float s_red[kWavesPerBlock];
    const int lane = threadIdx.x & (kWave - 1);

    const int64_t wave = (int64_t)__builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock + threadIdx.x / kWave);
    const int64_t rb = wave * a.rows_per_wave;
    const int64_t re = min(a.n, rb + a.rows_per_wave);
    float* ylds = s_y[threadIdx.x / kWave];
    half2v xr[GPL][16];
    StepBuf b0, b1;
    if constexpr (LPR * GPL <= 256) {
        // x (and the prologue's second operand) is loaded first and the first
        // two weight steps right after it: the weights are then in flight
        // while x is rearranged and the prologue computed, and waiting for x
        // never waits for them (the load counter retires in issue order).
        // Waves past the matrix take part in the prologue's barriers; their
        // loads read zeros.  Loads of steps past the wave's last one start
        // at row n, past the end of the codes and scales: they read zeros
        // without touching memory instead of another wave's rows.
        const int64_t steps = rb < a.n ? (re - rb + R - 1) / R : 0;
        const auto row_of = [&](int64_t st) { return st < steps ? rb + st * R : a.n; };
        const LinearRsrc rs = make_rsrc(a.packed, a.scales, (uint32_t)(a.n * a.ng * 2));
        if (a.prologue != WQ_PROLOGUE_NONE) {
            // 8-element chunks of x per thread for the longest row of this
            // shape (LPR GPL groups: the launcher picks a shape covering the
            // row), not of the largest K, to keep registers free for the
            // weight loads issued beside them.
            constexpr int CPT = (LPR * GPL * kGroup / 8 + kBlock - 1) / kBlock;
            stage_prologue<CPT>(a, s_x, s_red, [&] {
                issue_step<LPR, GPL, WQ_FUSED_CPOL, kFLoads>(b0, rs, row_of(0), a.ng, lane);
                issue_step<LPR, GPL, WQ_FUSED_CPOL, kFLoads>(b1, rs, row_of(1), a.ng, lane);
            });
            load_x_lane_lds<LPR, GPL>(s_x, a.ng, lane, xr);
        } else {
            u32x4 raw[GPL][4];
            load_x_raw<LPR, GPL, GPL>(a.x, a.ng, lane, raw);
            load_order_fence();
            issue_step<LPR, GPL, WQ_FUSED_CPOL, kFLoads>(b0, rs, row_of(0), a.ng, lane);
            issue_step<LPR, GPL, WQ_FUSED_CPOL, kFLoads>(b1, rs, row_of(1), a.ng, lane);
            pair_x<LPR, GPL, GPL>(raw, a.ng, lane, xr);
        }
        if (rb >= a.n) return;
        // As in gemv_m1_kernel: unconditional issues, so the wait counts
        // stay exact.
        for (int64_t s = 0; s < steps; s += 2) {
            const int64_t ra = rb + s * R;
            compute_step_f32<LPR, GPL, kFLoads>(b0, xr, (int)min((int64_t)R, re - ra), ylds, (int)(s * R), lane);
            issue_step<LPR, GPL, WQ_FUSED_CPOL, kFLoads>(b0, rs, row_of(s + 2), a.ng, lane);
            const int64_t rbb = ra + R;
            if (s + 1 < steps)
                compute_step_f32<LPR, GPL, kFLoads>(b1, xr, (int)min((int64_t)R, re - rbb), ylds, (int)((s + 1) * R), lane);
            issue_step<LPR, GPL, WQ_FUSED_CPOL, kFLoads>(b1, rs, row_of(s + 3), a.ng, lane);
        }
    } else {
        // Rows of more than 256 groups: x first, then the weights (their x
        // and weight registers together would cost waves per SIMD).  The
        // loop starts two steps early so that the first pass only issues and
        // every load comes from the same two issue sites.
        if (a.prologue != WQ_PROLOGUE_NONE) {
            stage_prologue<kMaxK / 8 / kBlock>(a, s_x, s_red, [] {});
            load_x_lane_lds<LPR, GPL>(s_x, a.ng, lane, xr);
        } else {
            load_x_lane<LPR, GPL, GPL>(a.x, a.ng, lane, xr);
        }
        if (rb >= a.n) return;
        const int64_t steps = (re - rb + R - 1) / R;
        const auto row_of = [&](int64_t st) { return st < steps ? rb + st * R : a.n; };
        const LinearRsrc rs = make_rsrc(a.packed, a.scales, (uint32_t)(a.n * a.ng * 2));
        for (int64_t s = -2; s < steps; s += 2) {
            const int64_t ra = rb + s * R;
            if (s >= 0) compute_step_f32<LPR, GPL, kFLoads>(b0, xr, (int)min((int64_t)R, re - ra), ylds, (int)(s * R), lane);
            issue_step<LPR, GPL, WQ_FUSED_CPOL, kFLoads>(b0, rs, row_of(s + 2), a.ng, lane);
            const int64_t rbb = ra + R;
            if (s + 1 >= 0 && s + 1 < steps)
                compute_step_f32<LPR, GPL, kFLoads>(b1, xr, (int)min((int64_t)R, re - rbb), ylds, (int)((s + 1) * R), lane);
            issue_step<LPR, GPL, WQ_FUSED_CPOL, kFLoads>(b1, rs, row_of(s + 3), a.ng, lane);
        }
    }
    flush_y_residual(a.y, a.residual, rb, ylds, (int)(re - rb), lane);
}

// (value, index) pairs: a larger value wins, then a smaller index; index -1
// (nothing seen, or only NaN) loses to anything.
__device__ __forceinline__ bool beats32(float v2, int i2, float v1, int i1) {
    if (i2 < 0) return false;
    if (i1 < 0) return true;
    return v2 > v1 || (v2 == v1 && i2 < i1);
}

// Logits per thread: the scalar head before the first 16-byte boundary and
// the scalar tail, plus up to kArgVec 16-byte vectors (8 logits each), all
// loaded in one round trip.  A thread first takes the maximum of its vectors
// (fmaxf ignores NaN), then the first element equal to it, scanning vectors
// in increasing index order; the block then reduces the (value, index)
// pairs.  NaN never wins; -1 when every logit is NaN.
constexpr int kArgVec = 16;

__global__ __launch_bounds__(kArgThreads) void argmax_kernel(const uint16_t* y, int n, int32_t* out) {
    constexpr int kWaves = kArgThreads / kWave;
    __shared__ float s_v[kWaves];
    __shared__ int s_i[kWaves];
    const int tid = threadIdx.x;
    const WQ_GLOBAL uint16_t* src = gbl(y);
    const int head = min(n, (int)(((16 - (reinterpret_cast<uintptr_t>(y) & 15)) & 15) / 2));
    const int nv = (n - head) / 8;
    const int tail0 = head + nv * 8;
    float best = 0.0f;
    int bi = -1;
    for (int v0 = tid; v0 < nv; v0 += kArgThreads * kArgVec) {
        u32x4 d[kArgVec];
        const WQ_GLOBAL u32x4* vec = reinterpret_cast<const WQ_GLOBAL u32x4*>(src + head);
#pragma unroll
        for (int u = 0; u < kArgVec; ++u) {
            const int v = v0 + u * kArgThreads;
            d[u] = v < nv ? vec[v] : u32x4{0x7E007E00u, 0x7E007E00u, 0x7E007E00u, 0x7E007E00u};  // NaN
        }
        float vmax[kArgVec];
        float m = __builtin_nanf("");
#pragma unroll
        for (int u = 0; u < kArgVec; ++u) {
            const uint32_t w[4] = {d[u].x, d[u].y, d[u].z, d[u].w};
            float t = __builtin_nanf("");   // stays NaN only for a vector of NaN
#pragma unroll
            for (int e = 0; e < 4; ++e) t = fmaxf(t, fmaxf(h2f(w[e] & 0xFFFFu), h2f(w[e] >> 16)));
            vmax[u] = t;
            m = fmaxf(m, t);
        }
        int found = -1;   // the first vector holding the maximum (none if all NaN)
#pragma unroll
        for (int u = kArgVec - 1; u >= 0; --u)
            if (vmax[u] == m) found = u;
        if (found >= 0) {
            u32x4 dv = d[0];
#pragma unroll
            for (int u = 1; u < kArgVec; ++u)
                if (u == found) dv = d[u];
            const uint32_t w[8] = {dv.x & 0xFFFFu, dv.x >> 16, dv.y & 0xFFFFu, dv.y >> 16,
                                   dv.z & 0xFFFFu, dv.z >> 16, dv.w & 0xFFFFu, dv.w >> 16};
            int e0 = -1;
#pragma unroll
            for (int e = 7; e >= 0; --e)
                if (h2f(w[e]) == m) e0 = e;
            const int idx = head + 8 * (v0 + found * kArgThreads) + e0;
            if (e0 >= 0 && beats32(m, idx, best, bi)) {
                best = m;
                bi = idx;
            }
        }
    }
    if (tid < head) {
        const float v = h2f(src[tid]);
        if (v == v && beats32(v, tid, best, bi)) {
            best = v;
            bi = tid;
        }
    }
    if (tail0 + tid < n) {
        const float v = h2f(src[tail0 + tid]);
        if (v == v && beats32(v, tail0 + tid, best, bi)) {
            best = v;
            bi = tail0 + tid;
        }
    }
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        const float v2 = __shfl_xor(best, o);
        const int i2 = __shfl_xor(bi, o);
        if (beats32(v2, i2, best, bi)) {
            best = v2;
            bi = i2;
        }
    }
    if ((tid & (kWave - 1)) == 0) {
        s_v[tid / kWave] = best;
        s_i[tid / kWave] = bi;
    }
    __syncthreads();
    if (tid == 0) {
        float v = s_v[0];
        int i = s_i[0];
        for (int w = 1; w < kWaves; ++w)
            if (beats32(s_v[w], s_i[w], v, i)) {
                v = s_v[w];
                i = s_i[w];
            }
        *out = i;
    }
}

// --------------------------------------------------- persistent dependent chain
//
// chain_kernel runs a whole dependent chain (one token's layers) in one
// cooperative launch: every workgroup stays resident, and no kernel
// boundary separates consecutive linears.  Two things make it pay:
//
//   * Weights depend on nothing, so each compute wave keeps issuing its next
//     steps across linear boundaries while it waits for the next x.
//   * Outputs move between workgroups as data that carries its own
//     validity: every output row is written to a library buffer T as one
//     32-bit word (fp16 value, 16-bit tag naming the linear and the launch)
//     with an agent-scope store, and a consumer reads its x (or residual)
//     from T with agent-scope loads until every word carries the tag it
//     expects.  A boundary thus costs a store and a load, not a store, its
//     acknowledgement, a flag, a poll and then the load.
//
// The caller's buffers are written only after the whole chain, by
// chain_epilogue (the final value of every output element, copied out of
// T), so no workgroup can overwrite an input that another still reads.
//
// Workgroup: eight compute waves (two per SIMD).  They own contiguous ranges
// of each linear's steps (the ranges of all waves of the grid, in order,
// cover the linear), stream them through NB register buffers in one
// sequence across linears, stage their rows' fp32 sums in LDS and write
// them to T when they move to the next linear.  x_eff of a linear is staged
// in LDS by the first four waves with fused_m1_kernel's prologue code and
// order, so results are bit-identical to one fused_m1_kernel launch per
// linear.  Every wait is bounded: a wait that runs past `timeout` clock
// ticks records the failure (per chain and in the device's error word) and
// every later wait of the launch gives up at once, so every wave ends.
constexpr int kChainWaves = 8;
constexpr int kChainPrologueWaves = kWavesPerBlock;  // the waves that stage x_eff (256 threads)
constexpr int kChainThreads = kChainWaves * kWave;
constexpr int kChainMaxK = 8192;      // rows of up to 256 groups
constexpr int kChainWaveRows = 512;   // rows of one linear a wave stages
constexpr uint32_t kChainOut = 0x80000000u;  // offset of unused load slots: past every chain buffer
constexpr uint32_t kChainTagPeriod = 32767;  // tags 1..32767; 0 marks nothing written

// Cache policy of an agent-scope access (sc1): coherent between the chip's
// L2 caches, as relaxed agent-scope atomics are.
constexpr int kCpolAgent = 16;

// Rows per slot of a step: as many as fill `loads` loads.
__host__ __device__ constexpr int chain_u(int gpl, int loads) { return gpl >= loads ? 1 : loads / gpl; }

// One linear of a chain as the kernel reads it.
struct ChainLinear {
    const void* packed;
    const uint16_t* scales;
    const uint16_t* x;         // the caller's x, when x_t < 0
    const uint16_t* norm;
    const uint16_t* residual;  // the caller's residual, when res_t < 0 (null: none)
    int64_t n;
    int64_t steps;             // ceil(n / rows per step)
    int64_t x_t;               // word offset of x in T (an earlier linear's outputs), or -1
    int64_t res_t;             // word offset of the residual in T, or -1
    int64_t y_t;               // word offset of this linear's outputs in T
    int32_t x_lin, res_lin;    // the linears whose outputs x_t and res_t point into
    int32_t ng, lpr, gpl, u;
    int32_t prologue;
    float eps;
};
static_assert(sizeof(ChainLinear) == 112, "ChainLinear layout");

// A run of final output values: T[t, t + count) -> y[0, count).
struct ChainCopy {
    uint16_t* y;
    int64_t t;
    int64_t count;
};
static_assert(sizeof(ChainCopy) == 24, "ChainCopy layout");

// Per-chain control words (in the chain's library buffer, zeroed when the
// buffer is set up): [0] the launch epoch, [1] epoch + 1 of a launch that
// gave up.  The device's error word is what wq_fused_check reports.
static __device__ uint32_t chain_err_flag;

__device__ __forceinline__ uint32_t ld_agent(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint32_t chain_tag(uint32_t epoch, int lin) {
    return (epoch + (uint32_t)lin) % kChainTagPeriod + 1u;
}

// First step of compute wave gw (of `waves`) in a linear of `steps` steps.
__device__ __forceinline__ int64_t chain_step0(int64_t gw, int64_t steps, int64_t waves) { return gw * steps / waves; }

// Bounded waiting, shared by every wait of a launch: gives up once the wait
// has run past the limit or once any wave of the launch has given up.
struct ChainWait {
    uint32_t* ctl;
    uint32_t epoch;
    uint64_t timeout;
    __device__ __forceinline__ bool give_up(uint64_t t0) const {
        if (ld_agent(ctl + 1) == epoch + 1u) return true;
        if (__builtin_amdgcn_s_memrealtime() - t0 > timeout) {
            st_agent(ctl + 1, epoch + 1u);
            st_agent(&chain_err_flag, 1u);
            return true;
        }
        return false;
    }
};

// Issue side: walks the wave's steps in order across linears and issues each
// step's loads.  Every step issues LOADS code and LOADS scale loads whatever
// its shape, unused slots pointed past the buffer's end (they return zeros
// without a memory access), so every path issues the same loads and the
// compiler's wait counts stay exact.  Past the last linear the loads go to
// an empty buffer.
struct ChainIssue {
    int lin;          // linear being issued (== count: past the end)
    int64_t step, end;
    LinearRsrc r;
    uint32_t lane_w;  // this lane's byte offset within a step (codes; scales take 1/8)
    int ng, lpr, gpl, u, rows;  // rows per slot, rows per step
};

__device__ __forceinline__ void chain_issue_enter(ChainIssue& c, const ChainLinear* plan, int count, int64_t gw,
                                                  int64_t waves, int lane) {
    while (c.lin < count) {
        const ChainLinear& L = plan[c.lin];
        const int64_t sb = chain_step0(gw, L.steps, waves), se = chain_step0(gw + 1, L.steps, waves);
        if (sb < se) {
            c.step = sb;
            c.end = se;
            c.ng = L.ng;
            c.lpr = L.lpr;
            c.gpl = L.gpl;
            c.u = L.u;
            c.rows = L.u * (kWave / L.lpr);
            c.r = make_rsrc(L.packed, L.scales, (uint32_t)(L.n * L.ng * 2));
            const int slot = lane / c.lpr, sub = lane & (c.lpr - 1);
            c.lane_w = (uint32_t)(slot * L.u * L.ng + sub) * 16u;
            return;
        }
        ++c.lin;
    }
    c.step = c.end = 0;
    c.r.w = __builtin_amdgcn_make_buffer_rsrc(const_cast<ChainLinear*>(plan), (short)0, 0, kRawBufferFlags);
    c.r.s = c.r.w;
    c.lane_w = 0;
    c.ng = c.lpr = c.gpl = c.u = 1;
    c.rows = 1;
}

// Issue the step the cursor is at into b and move on; returns the step's
// linear (count past the end) and its step index in `step`.
template <int LOADS>
__device__ __forceinline__ int chain_issue(ChainIssue& c, StepBuf& b, int64_t& step, const ChainLinear* plan,
                                           int count, int64_t gw, int64_t waves, int lane) {
    const int lin = c.lin;
    step = c.step;
    const uint32_t g0 = (uint32_t)(c.step * c.rows * c.ng);
    const uint32_t lane_s = c.lane_w >> 3;
    const int nloads = lin < count ? c.gpl * c.u : 0;
    int u = 0, j = 0;
#pragma unroll
    for (int k = 0; k < LOADS; ++k) {
        const bool used = k < nloads;
        const uint32_t go = g0 + (uint32_t)(u * c.ng + c.lpr * j);
        const uint32_t sw = used ? go * 16u : kChainOut, ss = used ? go * 2u : kChainOut;
        b.w[k] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(c.r.w, c.lane_w, sw, kCpolNonTemporal));
        b.s[k] = __builtin_amdgcn_raw_buffer_load_b16(c.r.s, lane_s, ss, kCpolNonTemporal);
        if (++j == c.gpl) {
            j = 0;
            ++u;
        }
    }
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    if (lin < count && ++c.step >= c.end) {
        ++c.lin;
        chain_issue_enter(c, plan, count, gw, waves, lane);
    }
    return lin;
}

// compute_step_f32 for the chain's step shape (U rows per slot from chain_u).
template <int LPR, int GPL, int MAXG, int LOADS>
__device__ __forceinline__ void chain_compute(const StepBuf& b, const half2v (&xr)[MAXG][16], int nrows, float* ylds,
                                              int yrel, int lane) {
    constexpr int U = chain_u(GPL, LOADS);
    const int slot = lane / LPR;
    const int sub = lane & (LPR - 1);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        float acc = 0.0f;
#pragma unroll
        for (int j = 0; j < GPL; ++j) {
            const float s = h2f(b.s[u * GPL + j]);
            acc = fmaf(s, dot_group(b.w[u * GPL + j], xr[j]), acc);
        }
        const float tot = segment_sum<LPR>(acc);
        const int rr = slot * U + u;
        if (sub == LPR - 1 && rr < nrows) ylds[yrel + rr] = tot;
    }
}

// Eight consecutive values of a linear's outputs from T, as one 16-byte
// chunk of fp16 (two 16-byte loads of tagged words); `ok` when all eight
// carry `tag`.
__device__ __forceinline__ u32x4 chain_chunk(const __amdgpu_buffer_rsrc_t& rt, uint32_t word, uint32_t tag, bool& ok) {
    const u32x4 a = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rt, word * 4u, 0, kCpolAgent));
    const u32x4 b = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rt, word * 4u + 16u, 0, kCpolAgent));
    const uint32_t t = tag << 16;
    ok = ((a.x & 0xFFFF0000u) == t) && ((a.y & 0xFFFF0000u) == t) && ((a.z & 0xFFFF0000u) == t) &&
         ((a.w & 0xFFFF0000u) == t) && ((b.x & 0xFFFF0000u) == t) && ((b.y & 0xFFFF0000u) == t) &&
         ((b.z & 0xFFFF0000u) == t) && ((b.w & 0xFFFF0000u) == t);
    return u32x4{(a.x & 0xFFFFu) | (a.y << 16), (a.z & 0xFFFFu) | (a.w << 16), (b.x & 0xFFFFu) | (b.y << 16),
                 (b.z & 0xFFFFu) | (b.w << 16)};
}

// x_eff of linear L into LDS by the first 256 threads: stage_prologue's
// reduction order and arithmetic (so x_eff is bit-identical), x read either
// from the caller (external input) or from T, waiting until every word of
// it carries its producer's tag.  One workgroup barrier, two for RMSNorm;
// the other waves take the same number.
template <int CPT>
__device__ __forceinline__ void chain_prologue(const ChainLinear& L, const uint32_t* T, uint32_t epoch,
                                               const ChainWait& w, uint16_t* s_x, float* red) {
    const int tid = threadIdx.x;
    const int chunks = L.ng * (kGroup / 8);
    const bool two = L.prologue != WQ_PROLOGUE_NONE;
    const bool is_silu = L.prologue == WQ_PROLOGUE_SILU_MUL;
    const int xchunks = is_silu ? 2 * chunks : chunks;
    u32x4 xa[CPT], xb[CPT];
    if (L.x_t >= 0) {
        const __amdgpu_buffer_rsrc_t rt = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint32_t*>(T + L.x_t), (short)0, xchunks * 32, kRawBufferFlags);
        const uint32_t tag = chain_tag(epoch, L.x_lin);
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        bool done[CPT];
#pragma unroll
        for (int r = 0; r < CPT; ++r) done[r] = tid + r * kBlock >= chunks;
        for (;;) {
            bool all = true;
#pragma unroll
            for (int r = 0; r < CPT; ++r) {
                if (done[r]) continue;
                const int c = tid + r * kBlock;
                bool oka = true, okb = true;
                const u32x4 va = chain_chunk(rt, (uint32_t)c * 8u, tag, oka);
                u32x4 vb = va;
                if (is_silu) vb = chain_chunk(rt, (uint32_t)(chunks + c) * 8u, tag, okb);
                if (oka && okb) {
                    xa[r] = va;
                    if (is_silu) xb[r] = vb;
                    done[r] = true;
                }
                all = all && done[r];
            }
            if (__all(all)) break;
            if (w.give_up(t0)) break;
            __builtin_amdgcn_s_sleep(1);
        }
        if (L.prologue == WQ_PROLOGUE_RMSNORM) {
            const WQ_GLOBAL u32x4* ns = gbl(reinterpret_cast<const u32x4*>(L.norm));
#pragma unroll
            for (int r = 0; r < CPT; ++r)
                if (tid + r * kBlock < chunks) xb[r] = ns[tid + r * kBlock];
        }
    } else {
        const WQ_GLOBAL u32x4* xs = gbl(reinterpret_cast<const u32x4*>(L.x));
        const WQ_GLOBAL u32x4* bs = L.prologue == WQ_PROLOGUE_RMSNORM ? gbl(reinterpret_cast<const u32x4*>(L.norm))
                                                                      : xs + chunks;
#pragma unroll
        for (int r = 0; r < CPT; ++r) {
            const int c = tid + r * kBlock;
            if (c < chunks) {
                xa[r] = xs[c];
                if (two) xb[r] = bs[c];
            }
        }
    }
    float inv = 0.0f;
    if (L.prologue == WQ_PROLOGUE_RMSNORM) {
        float ss = 0.0f;
#pragma unroll
        for (int r = 0; r < CPT; ++r) {
            if (tid + r * kBlock >= chunks) continue;
            const uint32_t wv[4] = {xa[r].x, xa[r].y, xa[r].z, xa[r].w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float lo = h2f(wv[i] & 0xFFFFu), hi = h2f(wv[i] >> 16);
                ss = fmaf(lo, lo, ss);
                ss = fmaf(hi, hi, ss);
            }
        }
        const float total = block_sum(ss, red);
        inv = 1.0f / sqrtf(total / (float)(L.ng * kGroup) + L.eps);
    }
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
        const int c = tid + r * kBlock;
        if (c >= chunks) continue;
        if (!two) {
            reinterpret_cast<u32x4*>(s_x)[c] = xa[r];
            continue;
        }
        const uint32_t wa[4] = {xa[r].x, xa[r].y, xa[r].z, xa[r].w};
        const uint32_t wb[4] = {xb[r].x, xb[r].y, xb[r].z, xb[r].w};
        uint32_t o[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float v[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const float p = h2f(h ? wa[i] >> 16 : wa[i] & 0xFFFFu);
                const float q = h2f(h ? wb[i] >> 16 : wb[i] & 0xFFFFu);
                v[h] = L.prologue == WQ_PROLOGUE_RMSNORM ? (p * inv) * q : silu(p) * q;
            }
            o[i] = f2h(v[0]) | (f2h(v[1]) << 16);
        }
        reinterpret_cast<u32x4*>(s_x)[c] = u32x4{o[0], o[1], o[2], o[3]};
    }
    __syncthreads();
}

// This lane's x groups of a linear from x_eff in LDS (load_x_lane_lds with
// the shape known at run time, one code path for every shape so that xr is
// assigned in one place): group j < gpl of the lane's row slot, zero where
// the group index runs past the row and for j >= gpl.
template <int MAXG>
__device__ __forceinline__ void chain_x(const uint16_t* s_x, int ng, int lpr, int gpl, int lane,
                                        half2v (&xr)[MAXG][16]) {
    const int sub = lane & (lpr - 1);
#pragma unroll
    for (int j = 0; j < MAXG; ++j) {
        const bool act = j < gpl && sub + lpr * j < ng;
        const u32x4* src = reinterpret_cast<const u32x4*>(s_x + min(sub + lpr * j, ng - 1) * kGroup);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const u32x4 d = src[c];
            xr[j][4 * c + 0] = as_h2(act ? (d.x & 0xFFFFu) | (d.z << 16) : 0u);
            xr[j][4 * c + 1] = as_h2(act ? (d.x >> 16) | (d.z & 0xFFFF0000u) : 0u);
            xr[j][4 * c + 2] = as_h2(act ? (d.y & 0xFFFFu) | (d.w << 16) : 0u);
            xr[j][4 * c + 3] = as_h2(act ? (d.y >> 16) | (d.w & 0xFFFF0000u) : 0u);
        }
        // One group's raw vectors at a time: hoisting every group's LDS reads
        // ahead of the pairing would hold them all beside the buffers in flight.
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Write a wave's staged rows [r0, r1) of linear L to T (residual added, one
// rounding), tagged as linear `lin` of this launch.
__device__ __forceinline__ void chain_flush(const ChainLinear& L, int lin, uint32_t* T, uint32_t epoch,
                                            const ChainWait& w, const float* ylds, int64_t r0, int64_t r1,
                                            int lane) {
    wave_lds_sync();
    const uint32_t tag = chain_tag(epoch, lin) << 16;
    const uint32_t rtag = L.res_t >= 0 ? chain_tag(epoch, L.res_lin) : 0u;
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    for (int64_t r = r0 + lane; __any(r < r1); r += kWave) {
        const bool mine = r < r1;
        float v = mine ? ylds[r - r0] : 0.0f;
        if (L.res_t >= 0) {
            // The residual is an earlier linear's output: wait for its tag.
            uint32_t e = 0;
            bool ok = !mine;
            for (;;) {
                if (!ok) {
                    e = ld_agent(T + L.res_t + r);
                    ok = (e >> 16) == rtag;
                }
                if (__all(ok) || w.give_up(t0)) break;
                __builtin_amdgcn_s_sleep(1);
            }
            v += h2f(e & 0xFFFFu);
        } else if (L.residual && mine) {
            v += h2f(gbl(L.residual)[r]);
        }
        if (mine) st_agent(T + L.y_t + r, tag | f2h(v));
    }
    wave_lds_sync();
}

// Step shapes are coded lanes-per-row * 16 + groups-per-lane.  A kernel
// variant compiles the compute of the shapes in its list only: every extra
// shape in the dispatch raises the register pressure of all of them.
constexpr int chain_code(int lpr, int gpl) { return lpr * 16 + gpl; }

template <int MAXG, int LOADS, int... S>
__device__ __forceinline__ void chain_compute_any(int shape, const StepBuf& b, const half2v (&xr)[MAXG][16], int nrows,
                                                  float* ylds, int yrel, int lane) {
    ((shape == S ? (chain_compute<S / 16, S % 16, MAXG, LOADS>(b, xr, nrows, ylds, yrel, lane), 0) : 0), ...);
}

// A variant: MAXG groups of x per lane (the largest groups-per-lane of its
// shapes), LOADS code loads per step, NB steps in flight per wave, and its
// shapes S.
template <int MAXG, int LOADS, int NB, int... S>
__global__ __launch_bounds__(kChainThreads, 2) void chain_kernel(const ChainLinear* __restrict__ plan, int count,
                                                                 uint32_t* __restrict__ T, uint32_t* ctl,
                                                                 uint64_t timeout) {
    static_assert(NB == 2 || NB == 3, "chain pipeline depth");
    static_assert(LOADS <= 8, "a step buffer holds eight loads");
    static_assert(MAXG * kWave * kGroup <= kChainMaxK * 2, "x_eff of the widest row fits its LDS buffer");
    __shared__ __align__(16) uint16_t s_x[2][kChainMaxK];
    __shared__ __align__(16) float s_y[kChainWaves][kChainWaveRows];
    __shared__ float s_red[kWavesPerBlock];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t waves = (int64_t)gridDim.x * kChainWaves;
    const int64_t gw = (int64_t)blockIdx.x * kChainWaves + wave;
    ChainWait w;
    w.ctl = ctl;
    w.epoch = ld_agent(ctl);
    w.timeout = timeout;
    const uint32_t epoch = w.epoch;
    float* ylds = s_y[wave];

    ChainIssue ic;
    ic.lin = 0;
    chain_issue_enter(ic, plan, count, gw, waves, lane);
    // The register buffers, as separate variables so that nothing is
    // indexed at run time: each holds one step (its linear and step index).
    StepBuf b0, b1, b2;
    int l0, l1, l2 = count;
    int64_t s0, s1, s2 = 0;
    l0 = chain_issue<LOADS>(ic, b0, s0, plan, count, gw, waves, lane);
    l1 = chain_issue<LOADS>(ic, b1, s1, plan, count, gw, waves, lane);
    if constexpr (NB == 3) l2 = chain_issue<LOADS>(ic, b2, s2, plan, count, gw, waves, lane);

    half2v xr[MAXG][16];
    int cur = -1;            // linear whose x_eff is in xr
    int shape = 0;           // lpr * 16 + gpl of `cur`
    int64_t n = 0, rows = 1;
    int64_t wr0 = 0, wr1 = 0;  // this wave's rows of `cur`
    // Leave linear `cur` (write this wave's rows of it to T) and stage the
    // next one.
    auto advance = [&]() __attribute__((always_inline)) {
        if (cur >= 0) chain_flush(plan[cur], cur, T, epoch, w, ylds, wr0, wr1, lane);
        ++cur;
        if (cur >= count) return;
        const ChainLinear& L = plan[cur];
        uint16_t* sx = s_x[cur & 1];
        if (wave < kChainPrologueWaves) {
            chain_prologue<MAXG>(L, T, epoch, w, sx, s_red);
        } else {
            if (L.prologue == WQ_PROLOGUE_RMSNORM) __syncthreads();
            __syncthreads();
        }
        n = L.n;
        rows = L.u * (kWave / L.lpr);
        shape = L.lpr * 16 + L.gpl;
        wr0 = chain_step0(gw, L.steps, waves) * rows;
        wr1 = min(n, chain_step0(gw + 1, L.steps, waves) * rows);
        chain_x<MAXG>(sx, L.ng, L.lpr, L.gpl, lane, xr);
    };
    // Compute the step a buffer holds and refill it with the wave's next
    // step; false when the wave's steps are done.
    auto slot = [&](StepBuf& b, int& lin, int64_t& step) __attribute__((always_inline)) -> bool {
        if (lin >= count) return false;
        while (cur < lin) advance();
        const int64_t row = step * rows;
        const int nrows = (int)min(rows, n - row);
        chain_compute_any<MAXG, LOADS, S...>(shape, b, xr, nrows, ylds, (int)(row - wr0), lane);
        lin = chain_issue<LOADS>(ic, b, step, plan, count, gw, waves, lane);
        return true;
    };
    for (;;) {
        if (!slot(b0, l0, s0)) break;
        if (!slot(b1, l1, s1)) break;
        if constexpr (NB == 3)
            if (!slot(b2, l2, s2)) break;
    }
    while (cur < count) advance();
}

// After a chain: copy the final value of every output element from T to the
// caller's buffers (runs of T words that no later linear overwrites, so the
// copies are disjoint), then advance the chain's epoch.
__global__ __launch_bounds__(256) void chain_epilogue(const ChainCopy* __restrict__ copies, int ncopies,
                                                      const uint32_t* __restrict__ T, uint32_t* ctl, uint32_t count) {
    for (int i = blockIdx.x; i < ncopies; i += gridDim.x) {
        const ChainCopy c = copies[i];
        const WQ_GLOBAL uint32_t* src = gbl(T + c.t);
        WQ_GLOBAL uint16_t* dst = gbl(c.y);
        for (int64_t k = threadIdx.x; k < c.count; k += 256) dst[k] = (uint16_t)(src[k] & 0xFFFFu);
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) ctl[0] = ctl[0] + count;
}

// ------------------------------------------------------------------- host

template <int LPR, int GPL>
hipError_t launch_fused(const wq_fused_linear& l, hipStream_t stream) {
    constexpr int R = StepShape<LPR, GPL, kFLoads>::ROWS;
    const int64_t ng = l.K / kGroup;
    const int64_t steps = (l.N + R - 1) / R;
    const int64_t steps_per_wave = std::min((steps + kTargetWaves - 1) / kTargetWaves, (int64_t)(kYRows / R));
    Args a;
    a.packed = reinterpret_cast<const u32x4*>(l.packed_w);
    a.scales = l.scales;
    a.x = l.x;
    a.y = l.y;
    a.norm = l.norm_weight;
    a.residual = l.residual;
    a.n = l.N;
    a.rows_per_wave = steps_per_wave * R;
    a.ng = (int)ng;
    a.prologue = l.prologue;
    a.eps = l.eps;
    const int64_t waves = (l.N + a.rows_per_wave - 1) / a.rows_per_wave;
    const int64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
    const size_t lds = l.prologue == WQ_PROLOGUE_NONE ? 0 : (size_t)l.K * 2;
    hipLaunchKernelGGL((fused_m1_kernel<LPR, GPL>), dim3((unsigned)blocks), dim3(kBlock), lds, stream, a);
    return hipGetLastError();
}

hipError_t launch_one(const wq_fused_linear& l, hipStream_t stream) {
    int lpr = 64, gpl = 1;
    pick_shape((int)(l.K / kGroup), lpr, gpl);
#define WQ_FUSED_CASE(L, G) \
    if (lpr == L && gpl == G) return launch_fused<L, G>(l, stream);
    WQ_FUSED_CASE(64, 1) WQ_FUSED_CASE(64, 2) WQ_FUSED_CASE(64, 3) WQ_FUSED_CASE(64, 4)
    WQ_FUSED_CASE(64, 5) WQ_FUSED_CASE(64, 6) WQ_FUSED_CASE(64, 7) WQ_FUSED_CASE(64, 8)
    WQ_FUSED_CASE(32, 1) WQ_FUSED_CASE(32, 3) WQ_FUSED_CASE(32, 5) WQ_FUSED_CASE(32, 7)
    WQ_FUSED_CASE(16, 1) WQ_FUSED_CASE(16, 3) WQ_FUSED_CASE(16, 5) WQ_FUSED_CASE(16, 7)
#undef WQ_FUSED_CASE
    return hipErrorInvalidValue;  // pick_shape returns only the shapes above
}

wq_status err(wq_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
wq_status err(wq_status st, const char* fmt, ...) {
    char msg[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(msg, sizeof(msg), fmt, ap);
    va_end(ap);
    return record_error(st, msg);
}

bool aligned(const void* p, uintptr_t a) { return reinterpret_cast<uintptr_t>(p) % a == 0; }

struct Span {
    uintptr_t lo, hi;
};
Span span(const void* p, uint64_t bytes) {
    const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return Span{lo, lo + (uintptr_t)bytes};
}
bool overlaps(Span a, Span b) { return a.lo < a.hi && b.lo < b.hi && a.lo < b.hi && b.lo < a.hi; }

// Sorted, merged union of spans, for "does s overlap any of them".
struct SpanUnion {
    std::vector<Span> v;
    void build(std::vector<Span> in) {
        std::sort(in.begin(), in.end(), [](const Span& p, const Span& q) { return p.lo < q.lo; });
        for (const Span& s : in) {
            if (s.lo >= s.hi) continue;
            if (!v.empty() && s.lo <= v.back().hi) v.back().hi = std::max(v.back().hi, s.hi);
            else v.push_back(s);
        }
    }
    bool hits(Span s) const {
        auto it = std::lower_bound(v.begin(), v.end(), s.hi, [](const Span& p, uintptr_t x) { return p.lo < x; });
        return it != v.begin() && overlaps(*std::prev(it), s);
    }
};

wq_status check_linear(const char* fn, int64_t i, const wq_fused_linear& l) {
    if (!l.packed_w || !l.scales || !l.x || !l.y)
        return err(WQ_ERR_INVALID_ARG, "%s: linear %lld: null pointer", fn, (long long)i);
    if (l.prologue != WQ_PROLOGUE_NONE && l.prologue != WQ_PROLOGUE_RMSNORM && l.prologue != WQ_PROLOGUE_SILU_MUL)
        return err(WQ_ERR_INVALID_ARG, "%s: linear %lld: unknown prologue %d", fn, (long long)i, (int)l.prologue);
    if (l.prologue == WQ_PROLOGUE_RMSNORM) {
        if (!l.norm_weight) return err(WQ_ERR_INVALID_ARG, "%s: linear %lld: null norm_weight", fn, (long long)i);
        if (!std::isfinite(l.eps) || l.eps < 0.0f)
            return err(WQ_ERR_INVALID_ARG, "%s: linear %lld: eps must be finite and >= 0", fn, (long long)i);
    }
    if (l.N <= 0 || l.K <= 0 || l.N > WQ_MAX_N)
        return err(WQ_ERR_INVALID_ARG, "%s: linear %lld: N and K must be positive (N=%lld K=%lld)", fn, (long long)i,
                   (long long)l.N, (long long)l.K);
    if (l.K % kGroup != 0 || l.K > WQ_FUSED_MAX_K)
        return err(WQ_ERR_UNSUPPORTED, "%s: linear %lld: K must be a multiple of 32 up to %lld (K=%lld)", fn,
                   (long long)i, (long long)WQ_FUSED_MAX_K, (long long)l.K);
    if (!fits_rsrc(l.N, l.K / kGroup))
        return err(WQ_ERR_UNSUPPORTED, "%s: linear %lld: codes above 4 GiB", fn, (long long)i);
    if (!aligned(l.packed_w, 16) || !aligned(l.x, 16) ||
        (l.prologue == WQ_PROLOGUE_RMSNORM && !aligned(l.norm_weight, 16)))
        return err(WQ_ERR_MISALIGNED, "%s: linear %lld: packed_w, x and norm_weight must be 16-byte aligned", fn,
                   (long long)i);
    if (!aligned(l.scales, 2) || !aligned(l.y, 2) || !aligned(l.residual, 2))
        return err(WQ_ERR_MISALIGNED, "%s: linear %lld: scales, y and residual must be 2-byte aligned", fn,
                   (long long)i);
    const Span y = span(l.y, 2 * l.N);
    const int64_t xk = l.prologue == WQ_PROLOGUE_SILU_MUL ? 2 * l.K : l.K;
    if (overlaps(y, span(l.x, 2 * xk)))
        return err(WQ_ERR_INVALID_ARG, "%s: linear %lld: y overlaps x", fn, (long long)i);
    if (l.prologue == WQ_PROLOGUE_RMSNORM && overlaps(y, span(l.norm_weight, 2 * l.K)))
        return err(WQ_ERR_INVALID_ARG, "%s: linear %lld: y overlaps norm_weight", fn, (long long)i);
    if (l.residual && l.residual != l.y && overlaps(y, span(l.residual, 2 * l.N)))
        return err(WQ_ERR_INVALID_ARG, "%s: linear %lld: residual overlaps y without being y", fn, (long long)i);
    return WQ_OK;
}

// The compiled chain variants: the two step shapes of the Llama-class 3B
// layers (K = 3072 and 8192) on their own, then every narrow shape (rows of
// up to 256 groups).  A chain runs the first variant that has all of its
// shapes; other chains (rows of more than 256 groups, whose x alone would
// take 112 or more registers beside the buffers) take the per-linear path.
struct ChainVariant {
    const void* fn;
    int loads;
    int nshapes;
    int shapes[8];
};
#define WQ_C(L, G) chain_code(L, G)
#define WQ_NARROW WQ_C(64, 1), WQ_C(64, 2), WQ_C(64, 3), WQ_C(64, 4), WQ_C(32, 1), WQ_C(32, 3), WQ_C(16, 1), WQ_C(16, 3)
const ChainVariant kChainVariants[] = {
    {reinterpret_cast<const void*>(chain_kernel<4, 6, 3, WQ_C(32, 3), WQ_C(64, 4)>), 6, 2, {WQ_C(32, 3), WQ_C(64, 4)}},
    {reinterpret_cast<const void*>(chain_kernel<4, 6, 3, WQ_NARROW>), 6, 8, {WQ_NARROW}},
};
#undef WQ_NARROW
#undef WQ_C
constexpr int kChainVariantCount = sizeof(kChainVariants) / sizeof(kChainVariants[0]);

// Persistent-chain support of one device: whether cooperative launches work,
// how many workgroups of each variant run (one per CU), the clock rate.
struct ChainDevice {
    bool ready = false;
    bool coop = false;
    int blocks[kChainVariantCount] = {};
    uint64_t ticks_per_s = 0;
};
constexpr int kChainMaxDevices = 64;
std::mutex g_chain_mu;
ChainDevice g_chain_dev[kChainMaxDevices];

hipError_t chain_device(int device, ChainDevice*& out) {
    out = nullptr;
    if (device < 0 || device >= kChainMaxDevices) return hipSuccess;
    ChainDevice& d = g_chain_dev[device];
    if (!d.ready) {
        int coop = 0, cus = 0, rate_khz = 0;
        hipError_t e;
        if ((e = hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, device)) != hipSuccess) return e;
        if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device)) != hipSuccess) return e;
        if ((e = hipDeviceGetAttribute(&rate_khz, hipDeviceAttributeWallClockRate, device)) != hipSuccess) return e;
        for (int v = 0; v < kChainVariantCount; ++v) {
            int per = 0;
            if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kChainVariants[v].fn, kChainThreads, 0)) !=
                hipSuccess)
                return e;
            d.blocks[v] = per >= 1 ? cus : 0;
        }
        d.coop = coop != 0;
        d.ticks_per_s = (uint64_t)(rate_khz > 0 ? rate_khz : 100000) * 1000u;
        d.ready = true;
    }
    out = &d;
    return hipSuccess;
}

bool env_flag_off(const char* name) {
    const char* e = std::getenv(name);
    return e && e[0] == '0';
}

bool env_flag_on(const char* name) {
    const char* e = std::getenv(name);
    return e && e[0] == '1';
}

// The latest linear before `j` whose y overlaps [lo, hi): -2 when none does
// (the span is an input from outside the chain), -1 when the latest one does
// not hold all of it (not supported), else its index.
int chain_source(const std::vector<wq_fused_linear>& lin, int j, uintptr_t lo, uintptr_t hi) {
    for (int i = j - 1; i >= 0; --i) {
        const uintptr_t ylo = reinterpret_cast<uintptr_t>(lin[i].y), yhi = ylo + 2 * (uintptr_t)lin[i].N;
        if (ylo < hi && lo < yhi) return (ylo <= lo && hi <= yhi) ? i : -1;
    }
    return -2;
}

// Run the chain as one persistent cooperative launch (and its epilogue)
// when every linear fits the kernel's limits; `launched` is false (and
// nothing queued) when the chain must take the per-linear path instead.
wq_status launch_chain(const char* fn, const std::vector<wq_fused_linear>& lin, hipStream_t stream, bool& launched) {
    launched = false;
    if (!env_flag_on("WQ_FUSED_PERSISTENT")) return WQ_OK;
    const int count = (int)lin.size();
    if (count >= (int)kChainTagPeriod) return WQ_OK;
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return err(WQ_ERR_HIP, "%s: HIP error %d (%s)", fn, (int)e, hipGetErrorString(e));
    ChainDevice* cd = nullptr;
    {
        std::lock_guard<std::mutex> guard(g_chain_mu);
        if ((e = chain_device(device, cd)) != hipSuccess)
            return err(WQ_ERR_HIP, "%s: HIP error %d (%s)", fn, (int)e, hipGetErrorString(e));
    }
    if (!cd || !cd->coop) return WQ_OK;
    int variant = -1;
    for (int v = 0; v < kChainVariantCount && variant < 0; ++v) {
        bool all = true;
        for (const wq_fused_linear& l : lin) {
            int lpr = 64, gpl = 1;
            pick_shape((int)(l.K / kGroup), lpr, gpl);
            const int code = chain_code(lpr, gpl);
            bool found = false;
            for (int k = 0; k < kChainVariants[v].nshapes; ++k) found = found || kChainVariants[v].shapes[k] == code;
            all = all && found && l.K <= kChainMaxK;
        }
        if (all) variant = v;
    }
    if (variant < 0) return WQ_OK;
    const int loads = kChainVariants[variant].loads;
    int blocks = cd->blocks[variant];
    if (blocks < 1) return WQ_OK;
    // Tuning override: fewer workgroups than CUs.
    if (const char* env = std::getenv("WQ_CHAIN_BLOCKS")) {
        const int b = std::atoi(env);
        if (b > 0) blocks = std::min(blocks, b);
    }
    const int64_t waves = (int64_t)blocks * kChainWaves;
    // Descriptors: T offsets of every linear's outputs, and where each x and
    // residual comes from.
    std::vector<ChainLinear> cl(count);
    int64_t t_words = 0;
    for (int i = 0; i < count; ++i) {
        const wq_fused_linear& l = lin[i];
        ChainLinear& c = cl[i];
        int lpr = 64, gpl = 1;
        const int64_t ng = l.K / kGroup;
        pick_shape((int)ng, lpr, gpl);
        if (l.N * ng * 16 >= ((int64_t)1 << 31)) return WQ_OK;  // codes past the unused-slot offset
        const int u = chain_u(gpl, loads);
        const int64_t rows = (int64_t)u * (kWave / lpr);
        const int64_t steps = (l.N + rows - 1) / rows;
        if (((steps + waves - 1) / waves) * rows > kChainWaveRows) return WQ_OK;
        const uintptr_t xlo = reinterpret_cast<uintptr_t>(l.x);
        const int64_t xk = l.prologue == WQ_PROLOGUE_SILU_MUL ? 2 * l.K : l.K;
        const int xs = chain_source(lin, i, xlo, xlo + 2 * (uintptr_t)xk);
        if (xs == -1) return WQ_OK;
        int rs = -2;
        if (l.residual) {
            const uintptr_t rlo = reinterpret_cast<uintptr_t>(l.residual);
            rs = chain_source(lin, i, rlo, rlo + 2 * (uintptr_t)l.N);
            if (rs == -1) return WQ_OK;
        }
        if (l.prologue == WQ_PROLOGUE_RMSNORM) {
            // The norm weight must not be an output of the chain.
            const uintptr_t nlo = reinterpret_cast<uintptr_t>(l.norm_weight);
            if (chain_source(lin, count, nlo, nlo + 2 * (uintptr_t)l.K) != -2) return WQ_OK;
        }
        c = ChainLinear{};
        c.packed = l.packed_w;
        c.scales = l.scales;
        c.x = l.x;
        c.norm = l.norm_weight;
        c.residual = l.residual;
        c.n = l.N;
        c.steps = steps;
        c.y_t = t_words;
        t_words += l.N;
        c.x_lin = xs >= 0 ? xs : -1;
        c.x_t = xs >= 0 ? cl[xs].y_t + (int64_t)((xlo - reinterpret_cast<uintptr_t>(lin[xs].y)) / 2) : -1;
        c.res_lin = rs >= 0 ? rs : -1;
        c.res_t = rs >= 0 ? cl[rs].y_t + (int64_t)((reinterpret_cast<uintptr_t>(l.residual) -
                                                   reinterpret_cast<uintptr_t>(lin[rs].y)) / 2)
                          : -1;
        c.ng = (int32_t)ng;
        c.lpr = lpr;
        c.gpl = gpl;
        c.u = u;
        c.prologue = l.prologue;
        c.eps = l.eps;
    }
    // Final values: every output element comes from the last linear that
    // writes it, so the copies of the epilogue are disjoint.
    std::vector<ChainCopy> copies;
    {
        std::vector<Span> claimed;  // sorted, disjoint
        for (int i = count - 1; i >= 0; --i) {
            const uintptr_t lo = reinterpret_cast<uintptr_t>(lin[i].y), hi = lo + 2 * (uintptr_t)lin[i].N;
            uintptr_t p = lo;
            for (const Span& s : claimed) {
                if (s.hi <= p || s.lo >= hi) continue;
                if (s.lo > p) copies.push_back(ChainCopy{reinterpret_cast<uint16_t*>(p), cl[i].y_t + (int64_t)((p - lo) / 2),
                                                         (int64_t)((s.lo - p) / 2)});
                p = std::max(p, s.hi);
            }
            if (p < hi)
                copies.push_back(ChainCopy{reinterpret_cast<uint16_t*>(p), cl[i].y_t + (int64_t)((p - lo) / 2),
                                           (int64_t)((hi - p) / 2)});
            claimed.push_back(Span{lo, hi});
            std::sort(claimed.begin(), claimed.end(), [](const Span& a, const Span& b) { return a.lo < b.lo; });
            std::vector<Span> merged;
            for (const Span& s : claimed) {
                if (!merged.empty() && s.lo <= merged.back().hi) merged.back().hi = std::max(merged.back().hi, s.hi);
                else merged.push_back(s);
            }
            claimed.swap(merged);
        }
    }
    {
        // Runs of at most 4096 values, one workgroup each.
        std::vector<ChainCopy> split;
        for (const ChainCopy& c : copies)
            for (int64_t k = 0; k < c.count; k += 4096)
                split.push_back(ChainCopy{c.y + k, c.t + k, std::min<int64_t>(4096, c.count - k)});
        copies.swap(split);
    }
    const size_t lin_bytes = sizeof(ChainLinear) * count;
    std::vector<unsigned char> bytes(lin_bytes + sizeof(ChainCopy) * copies.size());
    std::memcpy(bytes.data(), cl.data(), lin_bytes);
    std::memcpy(bytes.data() + lin_bytes, copies.data(), sizeof(ChainCopy) * copies.size());
    // Zeroed library memory after the plan: the control words, then T.
    const size_t extra = 16 + (size_t)t_words * 4;
    const unsigned char* d_plan = nullptr;
    size_t extra_off = 0;
    bool capturing = false;
    const wq_status st = resident_plan(fn, stream, bytes, extra, d_plan, extra_off, capturing);
    // Under stream capture the chain takes the per-linear path: its launches
    // are plain kernel nodes.
    if (capturing) return WQ_OK;
    if (st != WQ_OK) return st;
    uint64_t timeout = cd->ticks_per_s / 2;  // half a second per wait
    if (const char* env = std::getenv("WQ_CHAIN_TIMEOUT_TICKS")) {
        const long long t = std::atoll(env);
        if (t > 0) timeout = (uint64_t)t;
    }
    const ChainLinear* plan = reinterpret_cast<const ChainLinear*>(d_plan);
    const ChainCopy* dcopies = reinterpret_cast<const ChainCopy*>(d_plan + lin_bytes);
    uint32_t* ctl = reinterpret_cast<uint32_t*>(const_cast<unsigned char*>(d_plan) + extra_off);
    uint32_t* T = ctl + 4;
    int cnt = count;
    void* args[] = {&plan, &cnt, &T, &ctl, &timeout};
    // WQ_CHAIN_COOPERATIVE=0 (for measurements) launches without the
    // co-residency guarantee; the bounded waits still end every wave.
    if (env_flag_off("WQ_CHAIN_COOPERATIVE"))
        e = hipLaunchKernel(kChainVariants[variant].fn, dim3(blocks), dim3(kChainThreads), args, 0, stream);
    else
        e = hipLaunchCooperativeKernel(kChainVariants[variant].fn, dim3(blocks), dim3(kChainThreads), args, 0, stream);
    if (e != hipSuccess) return err(WQ_ERR_HIP, "%s: HIP error %d (%s)", fn, (int)e, hipGetErrorString(e));
    const int ncopies = (int)copies.size();
    hipLaunchKernelGGL(chain_epilogue, dim3((unsigned)std::max(1, std::min(ncopies, 1024))), dim3(256), 0, stream,
                       dcopies, ncopies, T, ctl, (uint32_t)count);
    if ((e = hipGetLastError()) != hipSuccess)
        return err(WQ_ERR_HIP, "%s: HIP error %d (%s)", fn, (int)e, hipGetErrorString(e));
    launched = true;
    return WQ_OK;
}

}  // namespace
}  // namespace fused
}  // namespace wq

using namespace wq::fused;

extern "C" wq_status wq_fused_linears(const wq_fused_linear* linears, int64_t count, int32_t* argmax,
                                      int64_t group, void* stream) {
    static const char* fn = "wq_fused_linears";
    if (!linears) return err(WQ_ERR_INVALID_ARG, "%s: null descriptor array", fn);
    if (count <= 0 || count > WQ_MAX_LINEARS)
        return err(WQ_ERR_INVALID_ARG, "%s: count must be in [1, %lld] (count=%lld)", fn, (long long)WQ_MAX_LINEARS,
                   (long long)count);
    if (group != 32) return err(WQ_ERR_UNSUPPORTED, "%s: only group=32 is supported (got %lld)", fn, (long long)group);
    if (argmax && !aligned(argmax, 4)) return err(WQ_ERR_MISALIGNED, "%s: argmax must be 4-byte aligned", fn);
    std::vector<wq_fused_linear> lin(linears, linears + count);
    std::vector<Span> weights, all;
    for (int64_t i = 0; i < count; ++i) {
        const wq_status st = check_linear(fn, i, lin[i]);
        if (st != WQ_OK) return st;
        const wq_fused_linear& l = lin[i];
        weights.push_back(span(l.packed_w, l.N * l.K / 2));
        weights.push_back(span(l.scales, l.N * (l.K / kGroup) * 2));
    }
    SpanUnion wu;
    wu.build(weights);
    for (int64_t i = 0; i < count; ++i) {
        const wq_fused_linear& l = lin[i];
        if (wu.hits(span(l.y, 2 * l.N)))
            return err(WQ_ERR_INVALID_ARG, "%s: y of linear %lld overlaps packed_w or scales of a linear", fn,
                       (long long)i);
        if (argmax) {
            const int64_t xk = l.prologue == WQ_PROLOGUE_SILU_MUL ? 2 * l.K : l.K;
            all.push_back(span(l.x, 2 * xk));
            all.push_back(span(l.y, 2 * l.N));
            if (l.prologue == WQ_PROLOGUE_RMSNORM) all.push_back(span(l.norm_weight, 2 * l.K));
            if (l.residual) all.push_back(span(l.residual, 2 * l.N));
        }
    }
    if (argmax) {
        SpanUnion au;
        all.insert(all.end(), weights.begin(), weights.end());
        au.build(all);
        if (au.hits(span(argmax, 4))) return err(WQ_ERR_INVALID_ARG, "%s: argmax overlaps an array of the chain", fn);
    }
    (void)hipGetLastError();
    const hipStream_t s = static_cast<hipStream_t>(stream);
    bool launched = false;
    const wq_status cs = launch_chain(fn, lin, s, launched);
    if (cs != WQ_OK) return cs;
    for (int64_t i = 0; !launched && i < count; ++i) {
        const hipError_t e = launch_one(lin[i], s);
        if (e != hipSuccess)
            return err(WQ_ERR_HIP, "%s: linear %lld: HIP error %d (%s)", fn, (long long)i, (int)e, hipGetErrorString(e));
    }
    if (argmax) {
        const wq_fused_linear& last = lin[count - 1];
        hipLaunchKernelGGL(argmax_kernel, dim3(1), dim3(kArgThreads), 0, s, last.y, (int)last.N, argmax);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return err(WQ_ERR_HIP, "%s: argmax: HIP error %d (%s)", fn, (int)e, hipGetErrorString(e));
    }
    return WQ_OK;
}

extern "C" wq_status wq_fused_check(void* stream) {
    static const char* fn = "wq_fused_check";
    hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return err(WQ_ERR_HIP, "%s: HIP error %d (%s)", fn, (int)e, hipGetErrorString(e));
    uint32_t flag = 0;
    if ((e = hipMemcpyFromSymbol(&flag, HIP_SYMBOL(chain_err_flag), sizeof(flag), 0, hipMemcpyDeviceToHost)) != hipSuccess)
        return err(WQ_ERR_HIP, "%s: HIP error %d (%s)", fn, (int)e, hipGetErrorString(e));
    if (!flag) return WQ_OK;
    const uint32_t zero = 0;
    if ((e = hipMemcpyToSymbol(HIP_SYMBOL(chain_err_flag), &zero, sizeof(zero), 0, hipMemcpyHostToDevice)) != hipSuccess)
        return err(WQ_ERR_HIP, "%s: HIP error %d (%s)", fn, (int)e, hipGetErrorString(e));
    return err(WQ_ERR_HIP, "%s: a persistent chain on this device gave up: a wait between its workgroups ran past "
               "its time limit, and that call's outputs are undefined", fn);
}
