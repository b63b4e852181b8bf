// Small-batch 4-bit GEMM on the matrix cores: y[M][N] = x[M][K] dequant(W)^T
// for 2 <= M <= 16 per launch (the concurrent-sequences decode of the
// paper's serving engine, Sec. 2.2; GEMM tiling, Sec. 2.3).
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

// One step's loads: per weight-row tile u, this lane's 16-byte group and its
// scale; the four x pieces (one per group of the step) for this lane's batch
// row and word.
template <int U>
struct MStep {
    u32x4 w[U];
    uint32_t s[U];
    u32x4 xa[4];
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

// The unconditional loads of step `step` (groups 4 step .. 4 step + 3);
// group and row indices are clamped, so every address is valid.
template <int U>
__device__ __forceinline__ void issue_mstep(MStep<U>& b, const u32x4* packed, const uint16_t* scales,
                                            const uint16_t* xrow, const int64_t (&roff)[U], int step, int ng,
                                            int c) {
    const WQ_GLOBAL u32x4* gp = gbl(packed);
    const WQ_GLOBAL uint16_t* gs = gbl(scales);
    const int g = min(4 * step + c, ng - 1);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        b.w[u] = gp[roff[u] + g];
        b.s[u] = gs[roff[u] + g];
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const int gt = min(4 * step + t, ng - 1);
        b.xa[t] = *reinterpret_cast<const WQ_GLOBAL u32x4*>(gbl(xrow) + gt * kGroup + 8 * c);
    }
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// Multiply-accumulate one step into acc[u] (16 batch rows x 16 weight rows).
template <int U>
__device__ __forceinline__ void compute_mstep(const MStep<U>& b, float4v (&acc)[U], int step, int ng, int c) {
    // Operand A pieces: x[8c .. 8c + 8) of each group, reordered to the
    // dequantized codes' order (0, 4), (1, 5), (2, 6), (3, 7).
    half8 xa[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const u32x4 d = b.xa[t];
        u32x4 r;
        r.x = __builtin_amdgcn_perm(d.z, d.x, 0x05040100u);
        r.y = __builtin_amdgcn_perm(d.z, d.x, 0x07060302u);
        r.z = __builtin_amdgcn_perm(d.w, d.y, 0x05040100u);
        r.w = __builtin_amdgcn_perm(d.w, d.y, 0x07060302u);
        xa[t] = __builtin_bit_cast(half8, r);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        uint32_t w0 = b.w[u].x, w1 = b.w[u].y, w2 = b.w[u].z, w3 = b.w[u].w;
        transpose4(w0, w1, w2, w3);
        // Scale of this lane's row for group 4 step + c; zero past the row's
        // groups (the clamped codes then add nothing).
        uint32_t s0 = 4 * step + c < ng ? b.s[u] : 0u;
        uint32_t s1 = s0, s2 = s0, s3 = s0;
        transpose4(s0, s1, s2, s3);
        const uint32_t wt[4] = {w0, w1, w2, w3};
        const uint32_t st[4] = {s0, s1, s2, s3};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            half2v q[4];
            dequant_word(wt[t], q);
            // (q - 8) * s rounded once to fp16: the group's weights in the
            // scale of operand B, so the multiplies accumulate across groups.
            const uint32_t sp = (st[t] & 0xFFFFu) | (st[t] << 16);
            const half2v sc = as_h2(sp);
            const u32x4 qb = {__builtin_bit_cast(uint32_t, q[0] * sc), __builtin_bit_cast(uint32_t, q[1] * sc),
                              __builtin_bit_cast(uint32_t, q[2] * sc), __builtin_bit_cast(uint32_t, q[3] * sc)};
            acc[u] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa[t], __builtin_bit_cast(half8, qb), acc[u], 0, 0, 0);
        }
    }
}

template <int U, int W, int NB>
__global__ __launch_bounds__(64 * W) void gemm_mfma_kernel(const u32x4* packed, const uint16_t* scales,
                                                           const uint16_t* __restrict__ x,
                                                           uint16_t* __restrict__ y, int64_t n, int ng, int m) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int li = lane & 15, c = lane >> 4;
    const int64_t row0 = (int64_t)blockIdx.x * 16 * U;
    int64_t roff[U];
#pragma unroll
    for (int u = 0; u < U; ++u) roff[u] = min(row0 + 16 * u + li, n - 1) * ng;
    const uint16_t* xrow = x + (int64_t)min(li, m - 1) * ng * kGroup;
    const int nsteps = (ng + 3) / 4;
    const int sb = wave * nsteps / W, se = (wave + 1) * nsteps / W;

    float4v acc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) acc[u] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
    // Same loop shape as the batch-1 kernels: NB register buffers, starting
    // NB steps early so the first pass only issues; loads past the range
    // re-read its last step.
    MStep<U> buf[NB];
    const int last = max(se - 1, sb);
    for (int s = sb - NB; s < se; s += NB) {
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            if (s + i >= sb && s + i < se) compute_mstep<U>(buf[i], acc, s + i, ng, c);
            issue_mstep<U>(buf[i], packed, scales, xrow, roff, min(s + i + NB, last), ng, c);
        }
    }

    // Sum the W waves' partial tiles; wave 0 rounds and stores.
    __shared__ float red[W > 1 ? W : 1][U][4][kWave];
    if constexpr (W > 1) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int v = 0; v < 4; ++v) red[wave][u][v][lane] = acc[u][v];
        __syncthreads();
        if (wave != 0) return;
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float t = 0.0f;
                for (int w = 0; w < W; ++w) t += red[w][u][v][lane];
                acc[u][v] = t;
            }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t col = row0 + 16 * u + li;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int mr = 4 * c + v;
            if (mr < m && col < n) gbl(y)[mr * n + col] = __half_as_ushort(__float2half_rn(acc[u][v]));
        }
    }
}

template <int U, int W>
hipError_t launch_u_w(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y, int64_t n,
                      int64_t ng, int m, hipStream_t stream) {
    constexpr int NB = 3;
    const int64_t blocks = (n + 16 * U - 1) / (16 * U);
    hipLaunchKernelGGL((gemm_mfma_kernel<U, W, NB>), dim3((unsigned)blocks), dim3(64 * W), 0, stream,
                       reinterpret_cast<const u32x4*>(packed), scales, x, y, n, (int)ng, m);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_mfma(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y,
                            int64_t n, int64_t k, int64_t m, hipStream_t stream) {
    const int64_t ng = k / kGroup;
    const int64_t nsteps = (ng + 3) / 4;
    // Row tiles per block: as many (up to 4) as still leave 512 blocks, so a
    // wave's x loads serve several tiles; then waves per block (a split of
    // the row's groups) up to about 1024 waves, each keeping at least three
    // steps.  (Measured on the 8B shapes: more waves than that only add x
    // traffic.)
    int u = 4;
    while (u > 1 && (n + 16 * u - 1) / (16 * u) < 512) u /= 2;
    const int64_t blocks = (n + 16 * u - 1) / (16 * u);
    int w = 1;
    while (w < 16 && blocks * w * 2 <= 1024 && nsteps / (w * 2) >= 3) w *= 2;
    for (int64_t m0 = 0; m0 < m; m0 += 16) {
        const int mc = (int)std::min<int64_t>(16, m - m0);
        const uint16_t* xc = x + m0 * k;
        uint16_t* yc = y + m0 * n;
        hipError_t e = hipSuccess;
#define WQ_MFMA_CASE(U, W) \
    if (u == U && w == W) e = launch_u_w<U, W>(packed, scales, xc, yc, n, ng, mc, stream);
        WQ_MFMA_CASE(1, 1) WQ_MFMA_CASE(1, 2) WQ_MFMA_CASE(1, 4) WQ_MFMA_CASE(1, 8) WQ_MFMA_CASE(1, 16)
        WQ_MFMA_CASE(2, 1) WQ_MFMA_CASE(2, 2) WQ_MFMA_CASE(2, 4) WQ_MFMA_CASE(2, 8) WQ_MFMA_CASE(2, 16)
        WQ_MFMA_CASE(4, 1) WQ_MFMA_CASE(4, 2) WQ_MFMA_CASE(4, 4) WQ_MFMA_CASE(4, 8) WQ_MFMA_CASE(4, 16)
#undef WQ_MFMA_CASE
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace wq
