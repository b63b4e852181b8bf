// Small-batch 4-bit GEMM on the matrix cores: y[M][N] = x[M][K] dequant(W)^T
// for up to 16 batch rows per launch, used from M = 8 on (smaller batches
// run on the vector kernel).  Batching several sequences is this library's
// extension of the paper's batch-1 decoding; the tiling follows the
// operator-level GEMM tiling the paper's compiler applies (Sec. 2.3).
//
// One v_mfma_f32_16x16x32_f16 multiplies a 16 x 32 block of x (16 batch
// rows, one 32-element group) by the dequantized 32 x 16 block of W^T (the
// same group of 16 weight rows).  x is operand A, the weights operand B, so
// the 16 x 16 result holds, in every lane, four batch rows of ONE weight row.
// The codes are dequantized exactly (q - 8 in fp16), then multiplied by the
// group's scale and rounded once to fp16 (relative error at most 2^-11 per
// weight, so the result stays within half the 1e-3 * sum |w x| tolerance;
// |q - 8| * s must stay below the fp16 range, i.e. scales below 8188), and
// the multiplies accumulate in fp32 across all groups.  Lane layouts
// (checked on the device): A lane l holds
// A[l % 16][8 (l / 16) + v], B lane l holds B[8 (l / 16) + v][l % 16], and
// the result lane l holds D[4 (l / 16) + v][l % 16].
//
// Each lane loads one whole 16-byte group: lane l reads group g0 + l / 16 of
// weight row l % 16, four consecutive groups per 64-lane load.  A 4 x 4
// transpose across the four 16-lane rows (two permlane32 and two permlane16
// swaps) turns that into "word l / 16 of group g0 + t" in register t, which
// becomes operand B of the t-th multiply.  The scales go through the same
// transpose (four copies of one register) to give every lane the scale of its
// weight row for each of the four groups.
//
// Work split: a block owns 16 U weight rows; its W waves split the row's
// groups into W contiguous ranges of 4-group steps and are summed through LDS
// at the end.  Each wave streams its range through three register buffers
// (compute one step, refill that buffer with the step three ahead).
#include "wq_device.h"
#include "wq_internal.h"

namespace wq {
namespace {

using namespace dev;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float4v __attribute__((ext_vector_type(4)));

// One item's loads: this lane's 16-byte group of one weight-row tile at one
// step, and its scale.
struct MItem {
    u32x4 w;
    uint32_t s;
};

// Transpose 4 x 4 dwords held as register r in 16-lane row c (value M[c][r])
// into register t in row c holding M[t][c].
__device__ __forceinline__ void transpose4(uint32_t& a0, uint32_t& a1, uint32_t& a2, uint32_t& a3) {
    // Upper half of a0 <-> lower half of a2, and a1 <-> a3.
    auto p02 = __builtin_amdgcn_permlane32_swap(a0, a2, false, false);
    auto p13 = __builtin_amdgcn_permlane32_swap(a1, a3, false, false);
    a0 = p02[0]; a2 = p02[1];
    a1 = p13[0]; a3 = p13[1];
    // Odd rows of a0 <-> even rows of a1, and a2 <-> a3.
    auto q01 = __builtin_amdgcn_permlane16_swap(a0, a1, false, false);
    auto q23 = __builtin_amdgcn_permlane16_swap(a2, a3, false, false);
    a0 = q01[0]; a1 = q01[1];
    a2 = q23[0]; a3 = q23[1];
}

constexpr int kChunk = 4;   // steps of 4 groups whose x a wave holds at once (2 in some single-linear launches)
constexpr int kDepth = 8;   // items in flight per wave

// Issue item (tile tt, step s): rows row0 + 16 tt + (lane % 16), group
// 4 s + lane / 16.  The scalar offset carries everything wave-uniform; rows
// past N read zeros.
__device__ __forceinline__ void issue_item(MItem& b, const LinearRsrc& r, uint32_t lg, int64_t row0, int tt, int s,
                                           int ng) {
    const uint32_t go = (uint32_t)((row0 + 16 * tt) * ng + 4 * s);
    b.w = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r.w, lg * 16, go * 16, 0));
    b.s = __builtin_amdgcn_raw_buffer_load_b16(r.s, lg * 2, go * 2, 0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// Multiply-accumulate one item into acc (16 batch rows x the tile's 16 weight
// rows).  `valid`: the step lies in this wave's range and this lane's group
// in the row; otherwise the scale is zero and the item adds nothing.
__device__ __forceinline__ void compute_item(const MItem& b, const half8 (&xa)[4], float4v& acc, bool valid) {
    uint32_t w0 = b.w.x, w1 = b.w.y, w2 = b.w.z, w3 = b.w.w;
    transpose4(w0, w1, w2, w3);
    uint32_t s0 = valid ? b.s : 0u;
    uint32_t s1 = s0, s2 = s0, s3 = s0;
    transpose4(s0, s1, s2, s3);
    const uint32_t wt[4] = {w0, w1, w2, w3};
    const uint32_t st[4] = {s0, s1, s2, s3};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        half2v q[4];
        dequant_word(wt[t], q);
        // (q - 8) * s rounded once to fp16: the group's weights in the scale
        // of operand B, so the multiplies accumulate across groups.
        const half2v sc = as_h2((st[t] & 0xFFFFu) | (st[t] << 16));
        const u32x4 qb = {__builtin_bit_cast(uint32_t, q[0] * sc), __builtin_bit_cast(uint32_t, q[1] * sc),
                          __builtin_bit_cast(uint32_t, q[2] * sc), __builtin_bit_cast(uint32_t, q[3] * sc)};
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa[t], __builtin_bit_cast(half8, qb), acc, 0, 0, 0);
    }
}

// x for one step as operand A pieces: x[8c .. 8c + 8) of each of its four
// groups for batch row lane % 16, reordered to the dequantized codes' order
// (0, 4), (1, 5), (2, 6), (3, 7).  Groups past the row are clamped (their
// weights are masked).
__device__ __forceinline__ void load_x_step(const uint16_t* xrow, int s, int ng, int c, half8 (&xa)[4]) {
    u32x4 d[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const int g = min(4 * s + t, ng - 1);
        d[t] = *reinterpret_cast<const WQ_GLOBAL u32x4*>(gbl(xrow) + g * kGroup + 8 * c);
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        u32x4 r;
        r.x = __builtin_amdgcn_perm(d[t].z, d[t].x, 0x05040100u);
        r.y = __builtin_amdgcn_perm(d[t].z, d[t].x, 0x07060302u);
        r.z = __builtin_amdgcn_perm(d[t].w, d[t].y, 0x05040100u);
        r.w = __builtin_amdgcn_perm(d[t].w, d[t].y, 0x07060302u);
        xa[t] = __builtin_bit_cast(half8, r);
    }
}

// A block owns T tiles of 16 weight rows from row0 of one linear; its waves
// (blockDim / 64 of them) split the row's steps into contiguous ranges.  A
// wave takes its range in chunks of C steps: it loads the chunk's x
// once, then streams every tile's codes for those steps through a
// kDepth-item register pipeline.  The waves' partial tiles are summed through
// LDS in a fixed order and one wave per tile rounds and stores it.
template <int T, int C = kChunk>
__device__ __forceinline__ void mfma_block(const void* packed, const uint16_t* scales, const uint16_t* x,
                                           uint16_t* y, int64_t n, int ng, int m, int64_t row0) {
    constexpr int kItems = T * C;
    constexpr int kPre = kDepth < kItems ? kDepth : kItems;
    const int lane = threadIdx.x & (kWave - 1);
    const int nw = blockDim.x / kWave;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int li = lane & 15, c = lane >> 4;
    const int nsteps = (ng + 3) / 4;
    const int sb = wave * nsteps / nw, se = (wave + 1) * nsteps / nw;
    const LinearRsrc rs = make_rsrc(packed, scales, (uint32_t)(n * ng * 2));
    const uint32_t lg = (uint32_t)(li * ng + c);
    const uint16_t* xrow = x + (int64_t)min(li, m - 1) * ng * kGroup;

    float4v acc[T];
#pragma unroll
    for (int tt = 0; tt < T; ++tt) acc[tt] = float4v{0.0f, 0.0f, 0.0f, 0.0f};

    for (int c0 = sb; c0 < se; c0 += C) {
        MItem buf[kPre];
#pragma unroll
        for (int q = 0; q < kPre; ++q) issue_item(buf[q], rs, lg, row0, q / C, c0 + q % C, ng);
        half8 xa[C][4];
#pragma unroll
        for (int k = 0; k < C; ++k) load_x_step(xrow, min(c0 + k, nsteps - 1), ng, c, xa[k]);
#pragma unroll
        for (int q = 0; q < kItems; ++q) {
            const int tt = q / C, k = q % C, s = c0 + k;
            compute_item(buf[q % kPre], xa[k], acc[tt], s < se && 4 * s + c < ng);
            if (q + kPre < kItems)
                issue_item(buf[q % kPre], rs, lg, row0, (q + kPre) / C, c0 + (q + kPre) % C, ng);
        }
    }

    __shared__ float red[8][4][kWave];
    for (int tt = 0; tt < T; ++tt) {
        float4v mine = acc[0];
#pragma unroll
        for (int u = 1; u < T; ++u)
            if (u == tt) mine = acc[u];
        if (nw > 1) {
#pragma unroll
            for (int v = 0; v < 4; ++v) red[wave][v][lane] = mine[v];
            __syncthreads();
        }
        if (wave == tt % nw) {
            float4v tot = mine;
            if (nw > 1) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    float t = 0.0f;
                    for (int w = 0; w < nw; ++w) t += red[w][v][lane];
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
        if (nw > 1) __syncthreads();
    }
}

// One linear: block b owns rows [16 T b, 16 T (b + 1)).
template <int T, int C>
__global__ __launch_bounds__(512) void gemm_mfma_kernel(const void* packed, const uint16_t* scales,
                                                        const uint16_t* __restrict__ x, uint16_t* __restrict__ y,
                                                        int64_t n, int ng, int m) {
    mfma_block<T, C>(packed, scales, x, y, n, ng, m, (int64_t)blockIdx.x * 16 * T);
}

// Independent linears of a decode step in one launch: entry i owns blocks
// [first_step, first_step + steps) (its rows in 16 T-row tiles), found by
// binary search; batch rows [m0, m0 + m) of every linear.
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
    mfma_block<T>(e.packed, e.scales, e.x + m0 * k, e.y + m0 * e.n, e.n, e.ng, m,
                  (b - e.first_step) * 16 * T);
}

template <int T, int C>
hipError_t launch_t(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y, int64_t n,
                    int64_t ng, int m, int w, hipStream_t stream) {
    const int64_t blocks = (n + 16 * T - 1) / (16 * T);
    hipLaunchKernelGGL((gemm_mfma_kernel<T, C>), dim3((unsigned)blocks), dim3(64 * w), 0, stream, packed, scales, x,
                       y, n, (int)ng, m);
    return hipGetLastError();
}

}  // namespace

int grouped_mfma_tiles() { return 8; }

hipError_t launch_grouped_mfma(const DecodeEntry* entries, int count, int64_t blocks, int waves_per_block,
                               int64_t m0, int m, hipStream_t stream) {
    hipLaunchKernelGGL((grouped_mfma_kernel<8>), dim3((unsigned)blocks), dim3(64 * waves_per_block), 0, stream,
                       entries, count, m0, m);
    return hipGetLastError();
}

hipError_t launch_gemm_mfma(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y,
                            int64_t n, int64_t k, int64_t m, hipStream_t stream) {
    const int64_t ng = k / kGroup;
    const int64_t nsteps = (ng + 3) / 4;
    // Chunks of 2 steps (half the x registers, twice the waves per SIMD) for
    // the very tall and the very long linears, where that measured faster
    // (LM heads and K = 14336 at M = 8 and 16: about 12%); 4 elsewhere
    // (3B qkv and gate_up, 8B gate_up: 3-14% slower with 2).
    const int c = (n >= 65536 || ng >= 384) ? 2 : kChunk;
    // Waves per block: one chunk of steps each where K allows, at most 8.
    const int w = (int)std::min<int64_t>(8, (nsteps + c - 1) / c);
    // Tiles per block: as many (up to 8, sharing each x load) as still keep
    // about 1536 waves in flight.
    int t = 8;
    while (t > 1 && (n + 16 * t - 1) / (16 * t) * w < 1536) t /= 2;
    for (int64_t m0 = 0; m0 < m; m0 += 16) {
        const int mc = (int)std::min<int64_t>(16, m - m0);
        const uint16_t* xc = x + m0 * k;
        uint16_t* yc = y + m0 * n;
        hipError_t e = hipSuccess;
        switch (t * 10 + c) {
            case 84: e = launch_t<8, 4>(packed, scales, xc, yc, n, ng, mc, w, stream); break;
            case 44: e = launch_t<4, 4>(packed, scales, xc, yc, n, ng, mc, w, stream); break;
            case 24: e = launch_t<2, 4>(packed, scales, xc, yc, n, ng, mc, w, stream); break;
            case 14: e = launch_t<1, 4>(packed, scales, xc, yc, n, ng, mc, w, stream); break;
            case 82: e = launch_t<8, 2>(packed, scales, xc, yc, n, ng, mc, w, stream); break;
            case 42: e = launch_t<4, 2>(packed, scales, xc, yc, n, ng, mc, w, stream); break;
            case 22: e = launch_t<2, 2>(packed, scales, xc, yc, n, ng, mc, w, stream); break;
            default: e = launch_t<1, 2>(packed, scales, xc, yc, n, ng, mc, w, stream); break;
        }
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace wq
