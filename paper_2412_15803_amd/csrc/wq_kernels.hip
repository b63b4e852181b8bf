// Quantize+pack and single-linear GEMV kernels (gfx950, wave64).
#include "wq_device.h"
#include "wq_internal.h"

#include <cstdlib>

namespace wq {
namespace {

using namespace dev;

constexpr int kBlock = 256;  // 4 waves per workgroup
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kTargetWaves = 256 * 8;  // 256 CUs x 8 waves

// --------------------------------------------------------------- quantize
//
// One thread per (row, group), grid-stride.  Bit-exact: IEEE fp32 division
// (__fdiv_rn), round-to-nearest-even fp32->fp16 keeping subnormals, rintf
// (ties to even), clamp to [0, 15].
__global__ __launch_bounds__(kBlock) void pack_kernel(const float* __restrict__ w,
                                                      uint32_t* __restrict__ packed,
                                                      uint16_t* __restrict__ scales, int64_t n, int64_t k) {
    const int64_t ng = k / kGroup;
    const int64_t total = n * ng;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x; t < total; t += stride) {
        const int64_t row = t / ng;
        const int64_t g = t - row * ng;
        const float4* src = reinterpret_cast<const float4*>(w + row * k + g * kGroup);
        float v[kGroup];
#pragma unroll
        for (int i = 0; i < kGroup / 4; ++i) {
            const float4 f = src[i];
            v[4 * i + 0] = f.x;
            v[4 * i + 1] = f.y;
            v[4 * i + 2] = f.z;
            v[4 * i + 3] = f.w;
        }
        float amax = 0.0f;
#pragma unroll
        for (int i = 0; i < kGroup; ++i) amax = fmaxf(amax, fabsf(v[i]));
        const __half s16 = __float2half_rn(__fdiv_rn(amax, 7.0f));
        const float s = __half2float(s16);
        uint32_t words[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            uint32_t word = 0;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                uint32_t code = 8;
                if (s != 0.0f) {
                    const float q = rintf(__fdiv_rn(v[8 * j + i], s)) + 8.0f;
                    code = (uint32_t)fminf(fmaxf(q, 0.0f), 15.0f);
                }
                word |= code << (4 * i);
            }
            words[j] = word;
        }
        reinterpret_cast<uint4*>(packed)[row * ng + g] = make_uint4(words[0], words[1], words[2], words[3]);
        scales[row * ng + g] = __half_as_ushort(s16);
    }
}

// ------------------------------------------------------------ batch-1 GEMV
//
// Each wave owns a contiguous block of at most kYRows rows and walks it in
// steps through NB register buffers: compute buffer i, refill it with the
// step NB ahead, move to buffer i + 1.  Whenever the wave waits for a
// buffer, the other NB - 1 buffers' loads are in flight.  Outputs are staged
// in LDS and written once, after the last step.
//
// Launch shape and pipeline, as measured on the single linears of the 3B
// and 8B layers (cold weights): about 1024 waves (four per CU, in workgroups
// of four), steps of four 16-byte loads per lane (the decode step's kernel
// takes six), two buffers and the default cache policy.  Every change that
// put more loads in flight at once made these launches slower; 8B gate_up
// 28672x4096 took 15.1-15.3 us so, against 16.5 with six-load steps, 17.4-19.6
// with three to six buffers, and 18.2 (2048 waves) and 21.5 us (4096 waves)
// with six-load steps and two buffers.
#ifndef WQ_M1_STEP_LOADS
#define WQ_M1_STEP_LOADS 4
#endif
#ifndef WQ_M1_DEPTH
#define WQ_M1_DEPTH 2
#endif
#ifndef WQ_M1_CPOL
#define WQ_M1_CPOL kCpolNonTemporal
#endif
#ifndef WQ_M1_X_LDS
#define WQ_M1_X_LDS 0
#endif
#ifndef WQ_M1_WAVES
#define WQ_M1_WAVES (256 * 4)
#endif
constexpr int kM1Loads = WQ_M1_STEP_LOADS;
constexpr int kM1Waves = WQ_M1_WAVES;
static_assert(kM1Loads >= 1 && kM1Loads <= 8, "a step's loads fit StepBuf");

template <int LPR, int GPL>
__global__ __launch_bounds__(kBlock) void gemv_m1_kernel(const u32x4* packed, const uint16_t* scales,
                                                         const uint16_t* __restrict__ x,
                                                         uint16_t* __restrict__ y, int64_t n, int ng,
                                                         int64_t rows_per_wave) {
    constexpr int R = StepShape<LPR, GPL, kM1Loads>::ROWS;
    constexpr int NB = WQ_M1_DEPTH;
    const int lane = threadIdx.x & (kWave - 1);
    // Wave-uniform (the compiler cannot see that threadIdx.x / 64 is), so
    // the row bookkeeping stays in scalar registers and branches uniform.
    const int64_t wave = (int64_t)__builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock + threadIdx.x / kWave);
    const int64_t rb = wave * rows_per_wave;
#if !WQ_M1_X_LDS
    if (rb >= n) return;
#endif
    const int64_t re = min(n, rb + rows_per_wave);
    const int64_t steps = rb < n ? (re - rb + R - 1) / R : 0;
    const LinearRsrc rs = make_rsrc(packed, scales, (uint32_t)(n * ng * 2));

    __shared__ __align__(16) uint16_t s_y[kWavesPerBlock][kYRows];
    uint16_t* ylds = s_y[threadIdx.x / kWave];

    // x's loads first, then the first weight steps, then x is paired: the
    // weights are in flight during x's round trip, and since x's loads are
    // the oldest, waiting for them never waits for a weight load.
#if WQ_M1_X_LDS
    // Variant: x read once per workgroup into LDS (16-byte chunks, thread t
    // taking chunks t, t + 256, ...), then each wave's lanes read their
    // groups from there.  Every wave takes part in the barrier.
    constexpr int kXChunks = LPR * GPL * (kGroup / 8);
    constexpr int CPT = (kXChunks + kBlock - 1) / kBlock;
    __shared__ __align__(16) u32x4 s_xk[kXChunks];
    const int chunks = ng * (kGroup / 8);
    u32x4 xc[CPT];
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
        const int c = (int)threadIdx.x + kBlock * r;
        if (c < chunks) xc[r] = gbl(reinterpret_cast<const u32x4*>(x))[c];
    }
    load_order_fence();
#else
    u32x4 xraw[GPL][4];
    load_x_raw<LPR, GPL, GPL>(x, ng, lane, xraw);
    load_order_fence();
#endif

    // Every pass issues into every buffer, also past the wave's last step:
    // those loads start at row n, past the end of the codes and scales, and
    // read zeros without touching memory (for codes within a step of 4 GiB
    // the 32-bit offset can wrap to an in-range load, whose data is never
    // used).  Every path through the loop thus issues the same loads, so the
    // compiler's wait counts stay exact.
    StepBuf buf[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i)
        issue_step<LPR, GPL, WQ_M1_CPOL, kM1Loads>(buf[i], rs, i < steps ? rb + i * R : n, ng, lane);
#if WQ_M1_X_LDS
#pragma unroll
    for (int r = 0; r < CPT; ++r) {
        const int c = (int)threadIdx.x + kBlock * r;
        if (c < chunks) s_xk[c] = xc[r];
    }
    __syncthreads();
    if (rb >= n) return;
    u32x4 xraw[GPL][4];
    {
        const int sub = lane & (LPR - 1);
#pragma unroll
        for (int j = 0; j < GPL; ++j)
#pragma unroll
            for (int c = 0; c < 4; ++c) xraw[j][c] = s_xk[4 * min(sub + LPR * j, ng - 1) + c];
    }
#endif
    half2v xr[GPL][16];
    pair_x<LPR, GPL, GPL>(xraw, ng, lane, xr);
    // steps >= 1 here: a loop that tests first would let the compiler sink
    // x's loads behind that test, after the weight loads.
    int64_t s = 0;
    do {
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            const int64_t si = s + i;
            if (si < steps) {
                const int64_t ri = rb + si * R;
                compute_step<LPR, GPL, GPL, kM1Loads>(buf[i], xr, (int)min((int64_t)R, re - ri), ylds, (int)(si * R),
                                                      lane);
            }
            issue_step<LPR, GPL, WQ_M1_CPOL, kM1Loads>(buf[i], rs, si + NB < steps ? rb + (si + NB) * R : n, ng,
                                                       lane);
        }
        s += NB;
    } while (s < steps);
    flush_y(y, rb, ylds, (int)(re - rb), lane);
}

// ------------------------------------------------ small batches, vector ALUs
//
// For 2 <= M <= 8 batch rows per pass.  A wave owns rows [rb, re) (at most
// kMbRows) and walks the row's groups in tiles: either 64 groups, lane l
// taking group 64 kt + l of every row, or (when a row's group count is an odd
// multiple of 32, or below 32) 32 groups, lanes 0-31 and 32-63 then taking
// group 32 kt + l % 32 of two different row sets.  Per tile it loads x of
// its group for the MB batch rows into registers (pre-paired like the
// batch-1 kernels), then streams its rows kMbU (per row set) at a time
// through two register buffers (buffer-resource loads, as in the batch-1
// kernels).  The dot products of one step are reduced across the lanes of
// each row set in one transposed reduction, and one lane per sum adds it to
// fp32 partial sums in LDS; after the last tile the partials are rounded
// once to fp16.
constexpr int kMbRows = 256;
constexpr int kMbU = 4;
constexpr int kMbStep = 2 * kMbU;  // grouped plans: rows per wave are a multiple of a step of either tiling
// Waves a single small-batch linear aims for: one per SIMD (2 to 12% faster
// than the 2048-wave split at M = 2 on the 8B-class shapes, 512 and 2048
// slower).
#ifndef WQ_MB_SINGLE_WAVES
#define WQ_MB_SINGLE_WAVES (256 * 4)
#endif
constexpr int64_t kMbSingleWaves = WQ_MB_SINGLE_WAVES;

template <int MB>
struct MbBuf {
    u32x4 w[kMbU];
    uint32_t s[kMbU];
};

// Issue the loads of one step: rows row0 + h kMbU + u (u < kMbU) for each of
// the H row sets, the tile's T = 64 / H groups per row.  Lane l takes group
// T kt + l % T of row set l / T.
template <int MB, int H>
__device__ __forceinline__ void mb_issue(MbBuf<MB>& b, const LinearRsrc& r, int64_t row0, int kt, int ng,
                                         int lane) {
    constexpr int T = kWave / H;
    const uint32_t lg = (uint32_t)(lane % T + (lane / T) * kMbU * ng);  // relative to the step's first group
#pragma unroll
    for (int u = 0; u < kMbU; ++u) {
        const uint32_t go = (uint32_t)((row0 + u) * ng + T * kt);
        b.w[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r.w, lg * 16, go * 16, 0));
        b.s[u] = __builtin_amdgcn_raw_buffer_load_b16(r.s, lg * 2, go * 2, 0);
    }
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// Sum each of V per-lane values (V = 8, 16 or 32) over the lanes of each of
// the H row sets (64 lanes when H = 1, 32 when H = 2), leaving value
// j + r W (j < W, W = V / 4 when H = 1, V / 2 when H = 2) in lane 16 r + j;
// with H = 2, values from V on belong to the second row set.  Swap levels
// halve the values per register while folding lanes l, l + 32 (only when
// both halves hold the same rows) and then 16-lane rows 0 + 1 and 2 + 3
// together (v_permlane32_swap exchanges the upper 32 lanes of its first
// operand with the lower 32 of its second, v_permlane16_swap the odd 16-lane
// rows of the first with the even rows of the second); a 16-lane DPP sum
// finishes each register and W selects gather the results.  About 2.5
// operations per value instead of a 6-step reduction each.
template <int V, int H>
__device__ __forceinline__ float transpose_reduce(const float (&v)[V], int lane) {
    constexpr int V1 = H == 1 ? V / 2 : V;
    constexpr int W = V1 / 2;
    float s[V1];
    if constexpr (H == 1) {
#pragma unroll
        for (int j = 0; j < V1; ++j) {
            // (A non-const result: with `const auto` this compiler reads
            // element 0 for both elements of the returned pair.)
            auto p = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, v[j]),
                                                       __builtin_bit_cast(uint32_t, v[j + V1]), false, false);
            const uint32_t lo = p[0], hi = p[1];
            s[j] = __builtin_bit_cast(float, lo) + __builtin_bit_cast(float, hi);
        }
    } else {
#pragma unroll
        for (int j = 0; j < V1; ++j) s[j] = v[j];
    }
    float t[W];
#pragma unroll
    for (int j = 0; j < W; ++j) {
        auto q = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, s[j]),
                                                   __builtin_bit_cast(uint32_t, s[j + W]), false, false);
        const uint32_t even = q[0], odd = q[1];
        t[j] = segment_sum<16>(__builtin_bit_cast(float, even) + __builtin_bit_cast(float, odd));
    }
    float r = t[0];
#pragma unroll
    for (int j = 1; j < W; ++j) r = (lane & 15) == j ? t[j] : r;
    return r;
}

template <int MB, int H>
__device__ __forceinline__ void mb_compute(const MbBuf<MB>& b, const half2v (&xr)[MB][16], float* part,
                                           int rel, int nrows, int lane) {
    constexpr int V = kMbU * MB;  // (row, batch row) sums of one row set
    float v[V];
#pragma unroll
    for (int u = 0; u < kMbU; ++u) {
        float acc[MB];
        const uint32_t wd[4] = {b.w[u].x, b.w[u].y, b.w[u].z, b.w[u].w};
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            half2v q[4];
            dequant_word(wd[c], q);
#pragma unroll
            for (int i = 0; i < MB; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    acc[i] = c == 0 && e == 0 ? dot2_first(q[0], xr[i][0])
                                              : __builtin_amdgcn_fdot2(q[e], xr[i][4 * c + e], acc[i], false);
        }
        const float sc = __half2float(__ushort_as_half((uint16_t)b.s[u]));
#pragma unroll
        for (int i = 0; i < MB; ++i) v[u * MB + i] = sc * acc[i];
    }
    // One reduction for the whole step; lane 16 r + j then holds the sum of
    // value idx = j + r W: row set idx / V, row (idx % V) / MB of it, batch
    // row idx % MB.
    constexpr int W = H == 1 ? V / 4 : V / 2;
    const float tot = transpose_reduce<V, H>(v, lane);
    const int j = lane & 15;
    const int idx = j + (lane >> 4) * W;
    const int row = (idx / V) * kMbU + (idx % V) / MB, i = idx % MB;
    if (j < W && row < nrows) part[(rel + row) * MB + i] += tot;
}

// Rows [rb, re) of one linear (re - rb <= kMbRows), batch rows [0, m), in
// tiles of T = 64 / H groups and steps of H kMbU rows.  The steps of all
// tiles form one stream through the two buffers: the loads of a tile's first
// steps are issued while the previous tile's last steps are computed, and x
// of the next tile is loaded right after the last step that reads the
// current one, ahead of the next weight loads.  Waiting for x then waits for
// the other buffer's loads too (issued earlier, and needed next anyway), so
// a tile boundary costs the pipeline one step of depth, not a full drain.
//
// Only tiles [kt0, kt1) are taken when the row's K is split across waves;
// then the fp32 partials stay in `part` for the caller to sum, else they are
// rounded and written to y.
template <int MB, int H>
__device__ __forceinline__ void mb_range(const void* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y,
                                         int64_t n, int ng, int m, int64_t rb, int64_t re, float* part, int lane,
                                         int kt0, int kt1, bool write) {
    constexpr int T = kWave / H;
    constexpr int R = H * kMbU;
    const int nrow = (int)(re - rb);
    const int steps = (nrow + R - 1) / R;
    const LinearRsrc rs = make_rsrc(packed, scales, (uint32_t)(n * ng * 2));
    const int64_t k = (int64_t)ng * kGroup;
    for (int i = lane; i < nrow * MB; i += kWave) part[i] = 0.0f;
    wave_lds_sync();

    const int ntiles = kt1;
    const int total = (kt1 - kt0) * steps;
    half2v xr[MB][16];
    auto load_x = [&](int kt) {
        const int g = T * kt + lane % T;
        const bool act = g < ng;
#pragma unroll
        for (int i = 0; i < MB; ++i) {
            const int mi = min(i, m - 1);  // rows past m repeat the last one (never stored)
            load_x_group(x + mi * k + (int64_t)min(g, ng - 1) * kGroup, xr[i]);
#pragma unroll
            for (int e = 0; e < 16; ++e) xr[i][e] = act ? xr[i][e] : half2v{(_Float16)0.0f, (_Float16)0.0f};
        }
    };
    load_x(kt0);
    // Issue position (tile ki, step si) and compute position (kc, sc), both
    // wave-uniform.  Issues run two steps ahead and, past the last tile,
    // read groups beyond the rows (zeros past the end), never computed.
    int ki = kt0, si = 0, kc = kt0, sc = 0;
    auto issue_next = [&](MbBuf<MB>& buf) {
        mb_issue<MB, H>(buf, rs, rb + (int64_t)si * R, ki, ng, lane);
        if (++si == steps) si = 0, ++ki;
    };
    auto compute_next = [&](const MbBuf<MB>& buf) {
        mb_compute<MB, H>(buf, xr, part, sc * R, nrow - sc * R, lane);
        if (++sc == steps) {
            sc = 0;
            if (++kc < ntiles) load_x(kc);
        }
    };
    // Starts two steps early so that the first pass only issues and every
    // load comes from the same two issue sites.
    MbBuf<MB> a, b;
    for (int t = -2; t < total; t += 2) {
        if (t >= 0) compute_next(a);
        issue_next(a);
        if (t + 1 >= 0 && t + 1 < total) compute_next(b);
        issue_next(b);
    }
    wave_lds_sync();
    if (!write) return;
    for (int i = lane; i < nrow * MB; i += kWave) {
        const int r = i / MB, mi = i % MB;
        if (mi < m) gbl(y)[mi * n + rb + r] = __half_as_ushort(__float2half_rn(part[i]));
    }
    wave_lds_sync();  // the slice is free again
}

// Two row sets of 32-group tiles when that pads a row's groups less than
// 64-group tiles do (96 groups: three full tiles instead of one and a half).
template <int MB>
__device__ __forceinline__ void mb_range_any(const void* packed, const uint16_t* scales, const uint16_t* x,
                                             uint16_t* y, int64_t n, int ng, int m, int64_t rb, int64_t re,
                                             float* part, int lane, int split = 1, int ks = 0) {
    if (mb_two_sets(ng)) {
        const int nt = (ng + 31) / 32;
        mb_range<MB, 2>(packed, scales, x, y, n, ng, m, rb, re, part, lane, ks * nt / split, (ks + 1) * nt / split,
                        split == 1);
    } else {
        const int nt = (ng + 63) / 64;
        mb_range<MB, 1>(packed, scales, x, y, n, ng, m, rb, re, part, lane, ks * nt / split, (ks + 1) * nt / split,
                        split == 1);
    }
}

// One linear.  With split = 1 every wave owns rows_per_wave rows; with
// split = 2 or 4 the block's waves form 4 / split row runs, the `split`
// waves of a run take contiguous parts of the row's K tiles, and their fp32
// partials are summed through LDS in a fixed order before the one rounding
// (for linears with too few rows to give every SIMD waves of its own).
template <int MB>
__global__ __launch_bounds__(kBlock) void gemv_mb_kernel(const void* packed, const uint16_t* scales,
                                                         const uint16_t* __restrict__ x, uint16_t* __restrict__ y,
                                                         int64_t n, int ng, int m, int64_t rows_per_wave, int split) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wib = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int ks = wib % split;
    const int64_t run = (int64_t)blockIdx.x * (kWavesPerBlock / split) + wib / split;
    const int64_t rb = run * rows_per_wave;
    const int64_t re = min(n, rb + rows_per_wave);
    __shared__ float s_part[kWavesPerBlock][kMbRows * MB];
    if (split == 1) {
        if (rb < n) mb_range_any<MB>(packed, scales, x, y, n, ng, m, rb, re, s_part[wib], lane);
        return;
    }
    if (rb < n) mb_range_any<MB>(packed, scales, x, y, n, ng, m, rb, re, s_part[wib], lane, split, ks);
    __syncthreads();
    if (ks != 0 || rb >= n) return;
    const int nrow = (int)(re - rb);
    for (int i = lane; i < nrow * MB; i += kWave) {
        float t = s_part[wib][i];
        for (int j = 1; j < split; ++j) t += s_part[wib + j][i];
        const int r = i / MB, mi = i % MB;
        if (mi < m) gbl(y)[mi * n + rb + r] = __half_as_ushort(__float2half_rn(t));
    }
}

// Independent linears of a decode step in one launch: entry i owns waves
// [first_step, first_step + steps), each `pad` rows of it (found by binary
// search over the entries); batch rows [m0, m0 + m).
template <int MB>
__global__ __launch_bounds__(kBlock) void grouped_mb_kernel(const DecodeEntry* __restrict__ entries, int count,
                                                            int64_t waves, int64_t m0, int m) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t wave = (int64_t)__builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock + threadIdx.x / kWave);
    if (wave >= waves) return;
    int lo = 0, hi = count - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (entries[mid].first_step <= wave) lo = mid;
        else hi = mid - 1;
    }
    const DecodeEntry& e = entries[lo];
    const int64_t rb = (wave - e.first_step) * e.pad;
    const int64_t k = (int64_t)e.ng * kGroup;
    __shared__ float s_part[kWavesPerBlock][kMbRows * MB];
    mb_range_any<MB>(e.packed, e.scales, e.x + m0 * k, e.y + m0 * e.n, e.n, e.ng, m, rb, min(e.n, rb + e.pad),
                     s_part[threadIdx.x / kWave], lane);
}

template <int MB>
hipError_t launch_mb(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y, int64_t n,
                     int64_t ng, int m, hipStream_t stream) {
    // x is loaded once per K tile and wave, so the rows a wave owns set how
    // many weight bytes each x load serves (with 4 rows and 4 batch rows, x
    // is 3.5x the weight bytes).  So: as many rows per wave, in whole steps
    // of the row's tiling (4 rows with 64-group tiles, 8 with two row sets),
    // as leave about kMbSingleWaves waves once each row run's K tiles are
    // split over up to 4 waves (two tiles each at least).
    const int64_t r = mb_two_sets(ng) ? 2 * kMbU : kMbU;
    const int64_t steps = (n + r - 1) / r;
    const int64_t ntiles = mb_two_sets(ng) ? (ng + 31) / 32 : (ng + 63) / 64;
    int64_t max_split = 1;
    while (max_split < 4 && ntiles >= 2 * max_split) max_split *= 2;
    const int64_t spw = std::max<int64_t>(1, std::min<int64_t>(steps * max_split / kMbSingleWaves, kMbRows / r));
    const int64_t rows_per_wave = spw * r;
    const int64_t runs = (n + rows_per_wave - 1) / rows_per_wave;
    int split = 1;
    while (split < max_split && runs * split < kMbSingleWaves) split *= 2;
    const int64_t blocks = (runs * split + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL((gemv_mb_kernel<MB>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, packed, scales, x, y,
                       n, (int)ng, m, rows_per_wave, split);
    return hipGetLastError();
}

// ------------------------------------------------------- generic GEMV (any M)
//
// One wave per (row, chunk of up to MC batch rows), grid-stride; lanes stride
// over the row's groups and read x straight from global memory.  Covers the
// shapes the tuned kernels do not (M > 1, K > 16384 at M = 1).
template <int MC>
__global__ __launch_bounds__(kBlock) void gemv_generic_kernel(const u32x4* packed,
                                                              const uint16_t* scales,
                                                              const uint16_t* __restrict__ x,
                                                              uint16_t* __restrict__ y, int64_t n,
                                                              int64_t ng, int64_t m, int64_t mchunks) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t total = n * mchunks;
    const int64_t wave_stride = (int64_t)gridDim.x * kWavesPerBlock;
    const int64_t k = ng * kGroup;
    for (int64_t wave = (int64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; wave < total;
         wave += wave_stride) {
        const int64_t row = wave / mchunks;
        const int64_t m0 = (wave - row * mchunks) * MC;
        const int mcount = (int)min((int64_t)MC, m - m0);
        float acc[MC];
#pragma unroll
        for (int i = 0; i < MC; ++i) acc[i] = 0.0f;
        for (int64_t g = lane; g < ng; g += kWave) {
            const u32x4 wv = packed[row * ng + g];
            const float s = __half2float(__ushort_as_half(scales[row * ng + g]));
#pragma unroll
            for (int i = 0; i < MC; ++i) {
                if (i < mcount) {
                    half2v xg[16];
                    load_x_group(x + (m0 + i) * k + g * kGroup, xg);
                    acc[i] = fmaf(s, dot_group(wv, xg), acc[i]);
                }
            }
        }
#pragma unroll
        for (int i = 0; i < MC; ++i) {
            const float tot = segment_sum<kWave>(acc[i]);
            if (lane == kWave - 1 && i < mcount) y[(m0 + i) * n + row] = __half_as_ushort(__float2half_rn(tot));
        }
    }
}


template <int LPR, int GPL>
hipError_t launch_m1(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y,
                     int64_t n, int64_t ng, hipStream_t stream) {
    constexpr int R = StepShape<LPR, GPL, kM1Loads>::ROWS;
    const int64_t steps = (n + R - 1) / R;
    // At most kYRows rows per wave (its LDS staging of y); more waves than
    // the target when the matrix is taller than that allows.
    const int64_t steps_per_wave = min((steps + kM1Waves - 1) / kM1Waves, (int64_t)(kYRows / R));
    const int64_t rows_per_wave = steps_per_wave * R;
    const int64_t waves = (n + rows_per_wave - 1) / rows_per_wave;
    const int64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL((gemv_m1_kernel<LPR, GPL>), dim3((unsigned)blocks), dim3(kBlock), 0, stream,
                       reinterpret_cast<const u32x4*>(packed), scales, x, y, n, (int)ng, rows_per_wave);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_grouped_mb(const DecodeEntry* entries, int count, int64_t waves, int64_t m0, int m,
                             hipStream_t stream) {
    const int64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
    if (m <= 2)
        hipLaunchKernelGGL((grouped_mb_kernel<2>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, entries, count,
                           waves, m0, m);
    else if (m <= 4)
        hipLaunchKernelGGL((grouped_mb_kernel<4>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, entries, count,
                           waves, m0, m);
    else
        hipLaunchKernelGGL((grouped_mb_kernel<8>), dim3((unsigned)blocks), dim3(kBlock), 0, stream, entries, count,
                           waves, m0, m);
    return hipGetLastError();
}

hipError_t mb_target_waves(int m, int device, int64_t& waves) {
    int per_cu = 0, cus = 0;
    hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess) return e;
    if (m <= 2) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, grouped_mb_kernel<2>, kBlock, 0);
    else if (m <= 4) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, grouped_mb_kernel<4>, kBlock, 0);
    else e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, grouped_mb_kernel<8>, kBlock, 0);
    if (e != hipSuccess) return e;
    cus = cus > 0 ? cus : 1;
    // Several rounds of waves, not one: with every wave resident at once the
    // CUs that happen to hold more of them set the time, while later rounds
    // go to whichever CU frees up first.  32 per CU measured best or within
    // noise of it on the 3B and 8B decode steps (M = 2, 4, 7).
    waves = max((int64_t)(per_cu > 0 ? per_cu : 1) * cus * kWavesPerBlock, (int64_t)32 * cus);
    return hipSuccess;
}

int mb_rows_for_work(int64_t work, int64_t ng) {
    const int64_t ngp = mb_padded_groups(ng);
    const int64_t r = (work + ngp - 1) / ngp;
    return (int)min((int64_t)kMbRows, max((int64_t)kMbStep, (r + kMbStep - 1) / kMbStep * kMbStep));
}

bool use_matrix_cores(int64_t m) {
    const char* v = std::getenv("WQ_SMALL_BATCH_VECTOR");
    if (v && v[0] == '1') return false;
    int64_t min_m = kMatrixCoreMinM;
    if (const char* e = std::getenv("WQ_MATRIX_MIN_M")) {
        const long long t = std::atoll(e);
        if (t >= 2) min_m = t;
    }
    return m >= min_m;
}

hipError_t launch_pack(const float* w, uint32_t* packed, uint16_t* scales, int64_t n, int64_t k,
                       hipStream_t stream) {
    const int64_t threads = n * (k / kGroup);
    const int64_t blocks = min((threads + kBlock - 1) / kBlock, (int64_t)1 << 20);
    hipLaunchKernelGGL(pack_kernel, dim3((unsigned)blocks), dim3(kBlock), 0, stream, w, packed, scales, n, k);
    return hipGetLastError();
}

hipError_t launch_gemv(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y,
                       int64_t n, int64_t k, int64_t m, hipStream_t stream) {
    const int64_t ng = k / kGroup;
    if (m == 1 && ng <= 512 && fits_rsrc(n, ng)) {
        int lpr = 64, gpl = 1;
        pick_shape((int)ng, lpr, gpl);
#define WQ_M1_CASE(L, G) \
    if (lpr == L && gpl == G) return launch_m1<L, G>(packed, scales, x, y, n, ng, stream);
        WQ_M1_CASE(64, 1) WQ_M1_CASE(64, 2) WQ_M1_CASE(64, 3) WQ_M1_CASE(64, 4)
        WQ_M1_CASE(64, 5) WQ_M1_CASE(64, 6) WQ_M1_CASE(64, 7) WQ_M1_CASE(64, 8)
        WQ_M1_CASE(32, 1) WQ_M1_CASE(32, 3) WQ_M1_CASE(32, 5) WQ_M1_CASE(32, 7)
        WQ_M1_CASE(16, 1) WQ_M1_CASE(16, 3) WQ_M1_CASE(16, 5) WQ_M1_CASE(16, 7)
#undef WQ_M1_CASE
    }
    if (m >= 2 && m <= kMaxSmallBatchM && fits_rsrc(n, ng)) {
        // Matrix cores from 8 batch rows on (measured faster than the vector
        // kernel there); below that, or when asked to, the vector kernel in
        // passes of up to 8 rows.
        if (use_matrix_cores(m)) return launch_gemm_mfma(packed, scales, x, y, n, k, m, stream);
        for (int64_t m0 = 0; m0 < m; m0 += 8) {
            const int mc = (int)min((int64_t)8, m - m0);
            const uint16_t* xc = x + m0 * k;
            uint16_t* yc = y + m0 * n;
            const hipError_t e = mc <= 2   ? launch_mb<2>(packed, scales, xc, yc, n, ng, mc, stream)
                                 : mc <= 4 ? launch_mb<4>(packed, scales, xc, yc, n, ng, mc, stream)
                                           : launch_mb<8>(packed, scales, xc, yc, n, ng, mc, stream);
            if (e != hipSuccess) return e;
        }
        return hipSuccess;
    }
    // Prompt-sized batches: the tiled matrix-core GEMM.
    if (m > kMaxSmallBatchM && prefill_fits(n, k, m)) return launch_prefill(packed, scales, x, y, n, k, m, stream);
    constexpr int MC = 4;
    const int64_t mchunks = (m + MC - 1) / MC;
    const int64_t waves = n * mchunks;
    const int64_t blocks = min((waves + kWavesPerBlock - 1) / kWavesPerBlock, (int64_t)1 << 20);
    hipLaunchKernelGGL((gemv_generic_kernel<MC>), dim3((unsigned)blocks), dim3(kBlock), 0, stream,
                       reinterpret_cast<const u32x4*>(packed), scales, x, y, n, ng, m, mchunks);
    return hipGetLastError();
}

}  // namespace wq
