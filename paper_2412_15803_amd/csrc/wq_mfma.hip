// Small-batch 4-bit GEMM on the matrix cores: y[M][N] = x[M][K] dequant(W)^T
// for up to 16 batch rows per launch, used from M = 3 on (M = 2 runs on the
// vector kernel).  Batching several sequences is this library's
// extension of the paper's batch-1 decoding; the tiling follows the
// operator-level GEMM tiling the paper's compiler applies (Sec. 2.3).
//
// One v_mfma_f32_16x16x32_f16 multiplies a 16 x 32 block of x (16 batch
// rows) by a dequantized 32 x 16 block of W^T (16 weight rows).  x is
// operand A, the weights operand B, so the 16 x 16 result holds, in every
// lane, four batch rows of ONE weight row.  Lane layouts (checked on the
// device): A lane l holds A[l % 16][8 (l / 16) + v], B lane l holds
// B[8 (l / 16) + v][l % 16], and the result lane l holds
// D[4 (l / 16) + v][l % 16].
//
// The K order inside a step of four groups is permuted, identically for x
// and W, so that each lane holds whole groups: in the matrix-core layout,
// lane 16 c + li holds group 4 s + c of weight row li (four words), and the
// t-th multiply of the step takes word t of it, so its 32-long K slice is
// word t of each of the step's four groups.  Summed over t, every element of
// the four groups is counted once, and each lane needs exactly one scale.
// The codes are dequantized exactly (q - 8 in fp16), multiplied by the
// lane's scale and rounded once to fp16 (relative error at most 2^-11 per
// weight, so the result stays within half the 1e-3 * sum |w x| tolerance;
// |q - 8| * s must stay below the fp16 range, i.e. scales below 8188), and
// the multiplies accumulate in fp32 across all groups.  Operand A carries x
// in the same permuted order: for multiply t, lane 16 c + li holds elements
// 8 t .. 8 t + 7 of group 4 s + c of batch row li, reordered as the
// dequantized codes are, (0, 4), (1, 5), (2, 6), (3, 7).
//
// Loads do not use that layout.  The texture addresser's cost of a 16-byte
// load grows with the distinct cache lines each quad of four consecutive
// lanes touches: measured with L2-resident data, about 57 cycles per wave
// instruction when the four lanes of every quad read four different rows
// (as the matrix-core layout has them), against 20 when each quad reads 64
// contiguous bytes of one row; with the matrix-core layout the addresser was
// 96% busy and set the speed.  So codes, scales and x are loaded in the load
// layout, lane 4 li + c holding what lane 16 c + li needs (each quad reads
// one row), and one ds_bpermute per register moves them across.
//
// Work split: a block owns T tiles of 16 weight rows; its W waves split the
// row's steps into W contiguous ranges and are summed through LDS at the
// end.  A wave streams its range through a register pipeline of eight
// items (one tile at one step each); x of a step is loaded ahead of the
// step's weight loads, so it arrives with them and waiting for it never
// drains the pipeline.
#include "wq_device.h"
#include "wq_internal.h"

namespace wq {
namespace {

using namespace dev;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float4v __attribute__((ext_vector_type(4)));

// Where a lane's scales come from.  kScaleItem (any shape): one 2-byte load
// per item, moved to the matrix-core layout like the codes.  kScaleLds (rows
// of a multiple of eight groups, 16-byte aligned scales): each tile's scales
// for a window of four pairs of steps (16 rows x 64 bytes) go straight into
// LDS with one 16-byte-per-lane direct-to-LDS load, and each lane reads its
// own from there.  Per-item 2-byte loads touch 16 cache lines for 128 bytes
// and lose them from L1 before the next step reads the same lines: with them
// the whole kernel ran a third slower than with its scale loads removed.
constexpr int kScaleItem = 0;
constexpr int kScaleLds = 1;

// One item's loads: this lane's 16-byte group of one weight-row tile at one
// step, and (kScaleItem) its scale.
struct MItem {
    u32x4 w;
    uint32_t s;
};

// Issue item (tile tt, step s) in the load layout: lane 4 q + j reads group
// 4 s + j of row row0 + 16 tt + q, so each quad of lanes reads 64
// contiguous bytes of one row (`lg` is the lane's part of the offset).  The
// scalar offset carries everything wave-uniform; rows past N read zeros.
template <int SM>
__device__ __forceinline__ void issue_item(MItem& b, const LinearRsrc& r, uint32_t lg, int64_t row0, int tt, int s,
                                           int ng) {
    const uint32_t go = (uint32_t)((row0 + 16 * tt) * ng + 4 * s);
    b.w = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r.w, lg * 16, go * 16, 0));
    if constexpr (SM == kScaleItem) b.s = __builtin_amdgcn_raw_buffer_load_b16(r.s, lg * 2, go * 2, 0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// Move a load-layout register to the matrix-core layout: lane 16 c + li
// takes the value of lane 4 li + c (`baddr` is that lane's byte address).
__device__ __forceinline__ uint32_t to_mfma(uint32_t v, int baddr) {
    return (uint32_t)__builtin_amdgcn_ds_bpermute(baddr, (int)v);
}

// ------------------------------------------------------- scale windows
//
// A window is four pairs of steps (32 groups); a tile's window is 16 rows x
// 64 bytes, 1 KiB of LDS, written by one direct-to-LDS load in which lane
// 4 q + u lands at byte 16 (4 q + u) and fetches piece u ^ ((q / 4) % 4) (8
// groups) of row q: each quad still reads its row's 64 bytes, and the
// XOR spreads the rows that a read instruction touches over the LDS banks.
// A wave has two window slots: the loads of window w + 1 are issued when
// window w starts, into the slot that window w - 1 has finished with.
constexpr int kWinPairs = 4;
constexpr int kTileWinBytes = 16 * 64;

typedef __attribute__((address_space(3))) uint8_t lds_u8;

__device__ __forceinline__ void issue_scale_window(const __amdgpu_buffer_rsrc_t& rsc, lds_u8* slot, uint32_t lane_off,
                                                   int64_t row0, int tt, int g0, int ng) {
    const uint32_t so = (uint32_t)(((row0 + 16 * tt) * ng + g0) * 2);  // wave-uniform
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsc, slot + tt * kTileWinBytes, 16, lane_off, so, 0, 0);
}

// The lane's scale bits from LDS (byte address `addr`).  An LDS read the
// compiler sees after a direct-to-LDS load gets a wait for every load in
// flight (it cannot tell the window slots apart), so the read is written
// out here and ordered by data dependences instead:
//   * `w` (a code register of the item) passes through the read: the read
//     is issued once the item's codes have arrived, and their load was
//     issued after the window's scale load (loads retire in order);
//   * the code register that comes out is what the item's permutes take,
//     so they are issued after the read;
//   * lds_scale_ready() hands the scale on only together with a permuted
//     word: the compiler waits for that permute before using it, and LDS
//     operations of a wave complete in order, so the read has completed.
__device__ __forceinline__ uint32_t lds_scale_read(uint32_t addr, uint32_t& w) {
    uint32_t v;
    asm volatile("ds_read_u16 %0, %2" : "=&v"(v), "+v"(w) : "v"(addr) : "memory");
    return v;
}

__device__ __forceinline__ uint32_t lds_scale_ready(uint32_t v, uint32_t permuted) {
    asm volatile("" : "+v"(v) : "v"(permuted));
    return v;
}

// Multiply-accumulate one item into acc (16 batch rows x the tile's 16 weight
// rows): its codes move to the matrix-core layout (lane 16 c + li: row li,
// group 4 s + c), multiply t takes word t of the lane's group, and the
// lane's scale comes from the item (kScaleItem) or the LDS window at
// `saddr`.  `keep` is zero where the group lies past the row or the step
// past the wave's range: the scale is then zero and the item adds nothing.
template <int SM>
__device__ __forceinline__ void compute_item(const MItem& b, const half8 (&xa)[4], float4v& acc, uint32_t keep,
                                             int baddr, uint32_t saddr) {
    uint32_t w0 = b.w.x, sv = 0;
    if constexpr (SM == kScaleLds) sv = lds_scale_read(saddr, w0);
    const uint32_t wd[4] = {to_mfma(w0, baddr), to_mfma(b.w.y, baddr), to_mfma(b.w.z, baddr),
                            to_mfma(b.w.w, baddr)};
    if constexpr (SM == kScaleItem) sv = to_mfma(b.s, baddr) & 0xFFFFu;
    else sv = lds_scale_ready(sv, wd[0]);
    // (q - 8) * s rounded once to fp16: the weights in the scale of operand
    // B, so the multiplies accumulate across groups.
    const half2v sc = as_h2((sv | (sv << 16)) & keep);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        half2v q[4];
        dequant_word(wd[t], q);
        const u32x4 qb = {__builtin_bit_cast(uint32_t, q[0] * sc), __builtin_bit_cast(uint32_t, q[1] * sc),
                          __builtin_bit_cast(uint32_t, q[2] * sc), __builtin_bit_cast(uint32_t, q[3] * sc)};
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa[t], __builtin_bit_cast(half8, qb), acc, 0, 0, 0);
    }
}

// x of one step as loaded: in the load layout, lane 4 li + c holds the 64
// bytes of group 4 s + c of batch row li (a group past the row is clamped to
// the last one; its weights are masked).  Unpacked into operands only when
// the step's compute starts: unpacking right after the loads would make the
// wave wait for everything in flight before them.
struct XRaw {
    u32x4 d[4];
};

__device__ __forceinline__ void issue_x(XRaw& r, const uint16_t* xrow, int s, int ng, int c) {
    const int g = min(4 * s + c, ng - 1);
    const WQ_GLOBAL u32x4* src = reinterpret_cast<const WQ_GLOBAL u32x4*>(gbl(xrow) + (int64_t)g * kGroup);
#pragma unroll
    for (int t = 0; t < 4; ++t) r.d[t] = src[t];
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// Operand A of the step's four multiplies, in the matrix-core layout (lane
// 16 c + li: batch row li, group 4 s + c): for multiply t, elements
// 8 t .. 8 t + 7 of the lane's group, reordered to the dequantized codes'
// order (0, 4), (1, 5), (2, 6), (3, 7).
__device__ __forceinline__ void unpack_x(const XRaw& r, half8 (&xa)[4], int baddr) {
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        u32x4 d;
        d.x = to_mfma(r.d[t].x, baddr);
        d.y = to_mfma(r.d[t].y, baddr);
        d.z = to_mfma(r.d[t].z, baddr);
        d.w = to_mfma(r.d[t].w, baddr);
        u32x4 o;
        o.x = __builtin_amdgcn_perm(d.z, d.x, 0x05040100u);
        o.y = __builtin_amdgcn_perm(d.z, d.x, 0x07060302u);
        o.z = __builtin_amdgcn_perm(d.w, d.y, 0x05040100u);
        o.w = __builtin_amdgcn_perm(d.w, d.y, 0x07060302u);
        xa[t] = __builtin_bit_cast(half8, o);
    }
}

// LDS per wave: its two scale-window slots (kScaleLds), which afterwards hold
// its partial tiles (T x 1 KiB) for the block's sum; or, with per-item
// scales, only the partial tiles (when the block has several waves).
__host__ __device__ constexpr int wave_lds_bytes(int t, int sm) { return sm == kScaleLds ? 2 * t * kTileWinBytes : t * 1024; }
__host__ __device__ constexpr int block_lds_bytes(int t, int sm, int waves) {
    return sm == kScaleLds || waves > 1 ? waves * wave_lds_bytes(t, sm) : 0;
}

// A block owns T tiles of 16 weight rows from row0 of one linear; its waves
// (blockDim / 64 of them) split the row's steps, in pairs, into contiguous
// ranges.  A wave streams its range a pair of steps at a time: item
// j = 2 tt + h of a pair is tile tt at step 2 p + h, so the two items that
// read one 128-byte run of each row (eight groups) are issued back to back
// (issuing all tiles of one step before the next step's measured 1.5x
// slower).  kDepth register buffers (four) hold the items in flight: the
// two items of a tile are computed, then their buffers are refilled with
// the items kDepth on, so one to two tiles' pairs of loads are always in
// flight (eight buffers, the first version, were 1-4% slower on the 3B and
// 8B steps at M = 4, 8 and 16; two, 9-15% slower).  x
// of the next pair is loaded right after the current pair's x is unpacked,
// ahead of that pair's weight loads, and unpacked when the pair starts.
// Loads past the wave's range re-read its last pair (already in the caches)
// and are never used.  The waves' partial tiles are summed through LDS in a
// fixed order and one wave per tile rounds and stores it.  `lds` is the
// block's dynamic LDS, wave_lds_bytes(T, SM) per wave.
#ifndef WQ_MFMA_DEPTH
#define WQ_MFMA_DEPTH 4
#endif
constexpr int kDepth = WQ_MFMA_DEPTH;

template <int T, int SM>
__device__ __forceinline__ void mfma_block(const void* packed, const uint16_t* scales, const uint16_t* x,
                                           uint16_t* y, int64_t n, int ng, int m, int64_t row0, lds_u8* lds) {
    constexpr int kItems = 2 * T;
    constexpr int D = kItems < kDepth ? kItems : kDepth;  // buffers
    static_assert(kItems % D == 0 && D % 2 == 0, "a pair's items fill the buffers a whole number of times");
    const int lane = threadIdx.x & (kWave - 1);
    const int nw = blockDim.x / kWave;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    // Matrix-core layout (lane 16 c + li) and load layout (lane 4 lq + cq).
    const int li = lane & 15, c = lane >> 4;
    const int lq = lane >> 2, cq = lane & 3;
    const int baddr = 4 * (4 * li + c);
    const int npairs = (ng + 7) / 8;
    const int pb = wave * npairs / nw, pe = (wave + 1) * npairs / nw;
    const LinearRsrc rs = make_rsrc(packed, scales, (uint32_t)(n * ng * 2));
    const uint32_t lg = (uint32_t)(lq * ng + cq);
    const uint16_t* xrow = x + (int64_t)min(lq, m - 1) * ng * kGroup;
    lds_u8* wlds = lds + wave * wave_lds_bytes(T, SM);
    // Scale windows: this lane's part of a window load's offset (piece
    // cq ^ (lq / 4) % 4 of row lq), and of a read's LDS address (row li's 64
    // bytes, then the XOR-placed piece and the group's half inside it).
    const uint32_t win_lane_off = (uint32_t)((lq * ng + 8 * (cq ^ ((lq >> 2) & 3))) * 2);
    const uint32_t rd_lane = (uint32_t)(size_t)wlds + (uint32_t)(li * 64 + 2 * c);
    const uint32_t rd_xor = (uint32_t)(((li >> 2) & 3) * 16);

    float4v acc[T];
#pragma unroll
    for (int tt = 0; tt < T; ++tt) acc[tt] = float4v{0.0f, 0.0f, 0.0f, 0.0f};

    if (pb < pe) {
        if constexpr (SM == kScaleLds) {
#pragma unroll
            for (int tt = 0; tt < T; ++tt) issue_scale_window(rs.s, wlds, win_lane_off, row0, tt, 8 * pb, ng);
#pragma unroll
            for (int tt = 0; tt < T; ++tt)
                issue_scale_window(rs.s, wlds + T * kTileWinBytes, win_lane_off, row0, tt, 8 * (pb + kWinPairs), ng);
        }
        XRaw xr[2];
        MItem buf[D];
        issue_x(xr[0], xrow, 2 * pb, ng, cq);
        issue_x(xr[1], xrow, 2 * pb + 1, ng, cq);
#pragma unroll
        for (int j = 0; j < D; j += 2) {
            issue_item<SM>(buf[j], rs, lg, row0, j / 2, 2 * pb, ng);
            issue_item<SM>(buf[j + 1], rs, lg, row0, j / 2, 2 * pb + 1, ng);
        }
        for (int p = pb; p < pe; ++p) {
            // Scale window of this pair: slot (p - pb) / 4 % 2, piece (p - pb) % 4.
            const int pr = p - pb;
            const int slot = (pr / kWinPairs) & 1;
            uint32_t rd = 0;
            if constexpr (SM == kScaleLds) {
                if (pr % kWinPairs == 0 && pr > 0) {
                    // Window pr / 4 starts; the other slot's window is done:
                    // load the window after this one into it.
#pragma unroll
                    for (int tt = 0; tt < T; ++tt)
                        issue_scale_window(rs.s, wlds + (slot ^ 1) * T * kTileWinBytes, win_lane_off, row0, tt,
                                           8 * (p + kWinPairs), ng);
                }
                rd = rd_lane + (uint32_t)(slot * T * kTileWinBytes) + ((uint32_t)((pr % kWinPairs) * 16) ^ rd_xor);
            }
            half8 xa[2][4];
            unpack_x(xr[0], xa[0], baddr);
            unpack_x(xr[1], xa[1], baddr);
            const int pn = min(p + 1, pe - 1);
            issue_x(xr[0], xrow, 2 * pn, ng, cq);
            issue_x(xr[1], xrow, 2 * pn + 1, ng, cq);
            const uint32_t keep0 = 8 * p + c < ng ? 0xFFFFFFFFu : 0u;
            const uint32_t keep1 = 8 * p + 4 + c < ng ? 0xFFFFFFFFu : 0u;
#pragma unroll
            for (int j = 0; j < kItems; j += 2) {
                const int tt = j / 2;
                MItem& b0 = buf[j % D];
                MItem& b1 = buf[(j + 1) % D];
                compute_item<SM>(b0, xa[0], acc[tt], keep0, baddr, rd + tt * kTileWinBytes);
                compute_item<SM>(b1, xa[1], acc[tt], keep1, baddr, rd + tt * kTileWinBytes + 8);
                // The tile these buffers take next: tile (j + D) / 2 of this
                // pair, or of the next pair past the last tile.
                const int jn = j + D;
                const int tn = jn < kItems ? jn / 2 : (jn - kItems) / 2;
                const int sn = jn < kItems ? 2 * p : 2 * pn;
                issue_item<SM>(b0, rs, lg, row0, tn, sn, ng);
                issue_item<SM>(b1, rs, lg, row0, tn, sn + 1, ng);
            }
        }
        // Scale-window loads may still be writing LDS that the partial sums
        // reuse.
        if constexpr (SM == kScaleLds) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }

    // Partial tiles of every wave to its LDS ([tile][v][lane] floats), then
    // wave w sums and stores the tiles tt with tt % nw == w, waves in order.
    typedef __attribute__((address_space(3))) float lds_f32;
    auto red = [&](int w, int tt, int v) -> lds_f32* {
        return reinterpret_cast<lds_f32*>(lds + w * wave_lds_bytes(T, SM)) + (tt * 4 + v) * kWave + lane;
    };
    if (nw > 1) {
#pragma unroll
        for (int tt = 0; tt < T; ++tt)
#pragma unroll
            for (int v = 0; v < 4; ++v) *red(wave, tt, v) = acc[tt][v];
        __syncthreads();
    }
#pragma unroll
    for (int tt = 0; tt < T; ++tt) {
        if (tt % nw != wave) continue;
        float4v tot = acc[tt];
        if (nw > 1) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float t = 0.0f;
                for (int w = 0; w < nw; ++w) t += *red(w, tt, v);
                tot[v] = t;
            }
        }
        const int64_t col = row0 + 16 * tt + li;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int mr = 4 * c + v;
            if (mr < m && col < n) gbl(y)[mr * n + col] = __half_as_ushort(__float2half_rn(tot[v]));
        }
    }
}

// Whether a linear's scales can come through LDS windows: 16-byte aligned
// and a multiple of eight groups per row, so that every window load reads
// 16-byte aligned pieces.
__host__ __device__ inline bool lds_scales(const uint16_t* scales, int64_t ng) {
    return ng % 8 == 0 && (reinterpret_cast<uintptr_t>(scales) & 15) == 0;
}

extern __shared__ __align__(16) uint8_t s_dyn[];

// One linear: block b owns rows [16 T b, 16 T (b + 1)).
template <int T, int SM>
__global__ __launch_bounds__(512) void gemm_mfma_kernel(const void* packed, const uint16_t* scales,
                                                        const uint16_t* __restrict__ x, uint16_t* __restrict__ y,
                                                        int64_t n, int ng, int m) {
    mfma_block<T, SM>(packed, scales, x, y, n, ng, m, (int64_t)blockIdx.x * 16 * T, (lds_u8*)s_dyn);
}

// Independent linears of a decode step in one launch: entry i owns blocks
// [first_step, first_step + steps) (its rows in 16 T-row tiles), found by
// binary search; batch rows [m0, m0 + m) of every linear.  The launch gives
// every wave two scale-window slots; linears whose scales cannot use them
// take per-item scale loads.
template <int T>
__global__ __launch_bounds__(512) void grouped_mfma_kernel(const DecodeEntry* __restrict__ entries, int count,
                                                           int64_t m0, int m) {
    const int64_t b = blockIdx.x;
    int lo = 0, hi = count - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (entries[mid].first_step <= b) lo = mid;
        else hi = mid - 1;
    }
    const DecodeEntry& e = entries[lo];
    const int64_t k = (int64_t)e.ng * kGroup;
    const int64_t row0 = (b - e.first_step) * 16 * T;
    lds_u8* lds = (lds_u8*)s_dyn;
    if (lds_scales(e.scales, e.ng))
        mfma_block<T, kScaleLds>(e.packed, e.scales, e.x + m0 * k, e.y + m0 * e.n, e.n, e.ng, m, row0, lds);
    else
        mfma_block<T, kScaleItem>(e.packed, e.scales, e.x + m0 * k, e.y + m0 * e.n, e.n, e.ng, m, row0, lds);
}

template <int T>
hipError_t launch_t(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y, int64_t n,
                    int64_t ng, int m, int w, hipStream_t stream) {
    const int64_t blocks = (n + 16 * T - 1) / (16 * T);
    if (lds_scales(scales, ng))
        hipLaunchKernelGGL((gemm_mfma_kernel<T, kScaleLds>), dim3((unsigned)blocks), dim3(64 * w),
                           block_lds_bytes(T, kScaleLds, w), stream, packed, scales, x, y, n, (int)ng, m);
    else
        hipLaunchKernelGGL((gemm_mfma_kernel<T, kScaleItem>), dim3((unsigned)blocks), dim3(64 * w),
                           block_lds_bytes(T, kScaleItem, w), stream, packed, scales, x, y, n, (int)ng, m);
    return hipGetLastError();
}

// A single linear's launch (measured over the 3B and 8B decode shapes at
// M = 4, 8, 16, with every waves-per-block / tiles-per-block pair forced):
// - K is split among a block's waves, a power of two up to four, with at
//   least WQ_MFMA_SPLIT_STEPS steps each: blocks of three waves (the 3B
//   shapes at 8 steps a wave) were 5-11% slower than blocks of four.
// - Tiles per block: as many as keep WQ_MFMA_TARGET_WAVES waves, but two
//   while that leaves WQ_MFMA_MIN_WAVES; with one tile a step's x (up to 16
//   batch rows) serves only 16 weight rows.
// - One tile per block at most 8 batch rows and at least
//   WQ_MFMA_WIDE_MIN_STEPS steps: eight waves per block (8B down at M = 4
//   15.9 -> 13.3 us, 3B down 10.0 -> 8.5 us; at M = 16 four waves stay
//   faster).
#ifndef WQ_MFMA_SPLIT_STEPS
#define WQ_MFMA_SPLIT_STEPS 6
#endif
#ifndef WQ_MFMA_TARGET_WAVES
#define WQ_MFMA_TARGET_WAVES 1024
#endif
#ifndef WQ_MFMA_MIN_WAVES
#define WQ_MFMA_MIN_WAVES 640
#endif
#ifndef WQ_MFMA_WIDE_MIN_STEPS
#define WQ_MFMA_WIDE_MIN_STEPS 32
#endif
#ifndef WQ_MFMA_TILES
#define WQ_MFMA_TILES 8
#endif
constexpr int kGroupedTiles = WQ_MFMA_TILES;
constexpr int kSplitWaves = 4;      // waves that split K in a block
constexpr int kWideSplitWaves = 8;  // the same for one-tile single linears (the kernels take 512 threads)

}  // namespace

int grouped_mfma_tiles() { return kGroupedTiles; }

// Four waves' scale-window slots (16 KiB each with eight tiles) fill the
// 64 KiB a launch may ask for without raising its limit.
int grouped_mfma_max_waves() { return kSplitWaves; }

hipError_t launch_grouped_mfma(const DecodeEntry* entries, int count, int64_t blocks, int waves_per_block,
                               int64_t m0, int m, hipStream_t stream) {
    hipLaunchKernelGGL((grouped_mfma_kernel<kGroupedTiles>), dim3((unsigned)blocks), dim3(64 * waves_per_block),
                       block_lds_bytes(kGroupedTiles, kScaleLds, waves_per_block), stream, entries, count, m0, m);
    return hipGetLastError();
}

hipError_t launch_gemm_mfma(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y,
                            int64_t n, int64_t k, int64_t m, hipStream_t stream) {
    const int64_t ng = k / kGroup;
    const int64_t nsteps = (ng + 3) / 4;
    int w = 1;
    while (w < grouped_mfma_max_waves() && nsteps / (2 * w) >= WQ_MFMA_SPLIT_STEPS) w *= 2;
    auto waves = [&](int tiles) { return (n + 16 * tiles - 1) / (16 * tiles) * w; };
    int t = WQ_MFMA_TILES;
    while (t > 1 && waves(t) < WQ_MFMA_TARGET_WAVES && !(t == 2 && waves(2) >= WQ_MFMA_MIN_WAVES)) t /= 2;
    for (int64_t m0 = 0; m0 < m; m0 += 16) {
        const int mc = (int)std::min<int64_t>(16, m - m0);
        const int wc = t == 1 && mc <= 8 && nsteps >= WQ_MFMA_WIDE_MIN_STEPS ? kWideSplitWaves : w;
        const uint16_t* xc = x + m0 * k;
        uint16_t* yc = y + m0 * n;
        hipError_t e = hipSuccess;
        switch (t) {
            case 8: e = launch_t<8>(packed, scales, xc, yc, n, ng, mc, wc, stream); break;
            case 4: e = launch_t<4>(packed, scales, xc, yc, n, ng, mc, wc, stream); break;
            case 2: e = launch_t<2>(packed, scales, xc, yc, n, ng, mc, wc, stream); break;
            default: e = launch_t<1>(packed, scales, xc, yc, n, ng, mc, wc, stream); break;
        }
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace wq
