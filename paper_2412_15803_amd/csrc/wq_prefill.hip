// Prefill (many rows of x at once) 4-bit GEMM on the matrix cores:
// y[M][N] = x[M][K] dequant(W)^T for M above the small-batch range.  Prompt
// processing runs the same quantized linears over every prompt token; the
// tiling is the operator-level GEMM tiling the paper's compiler applies
// (Sec. 2.3), written for gfx950's v_mfma_f32_16x16x32_f16.
//
// Tiles.  A 256-thread block computes a 128 (x rows) x 128 (weight rows)
// tile of y over K in stages of 64.  Per stage every thread loads four
// 16-byte pieces of x and one 16-byte group of codes (32 weights) with its
// scale, then writes them to LDS: x as is, the codes dequantized (exact
// q - 8, then times the scale, rounded once to fp16 as on the small-batch
// matrix-core path).  Within every 8-element piece both operands are stored
// in the order (0, 4, 1, 5, 2, 6, 3, 7) in which a code word dequantizes, so
// the fragments read back from LDS line up without further shuffles.  LDS is
// double-buffered: the global loads of stage s + 1 are in flight while
// stage s is multiplied, and one barrier per stage separates writing a
// buffer from reading it.
//
// Waves.  The four waves form a 2 x 2 grid, each owning 64 x 64 of the tile:
// 4 x 4 accumulators of 16 x 16, i.e. 16 multiplies per 32-deep k step.
// Lane layouts (as on the small-batch path): A lane l holds
// A[l % 16][8 (l / 16) + v], B lane l holds B[8 (l / 16) + v][l % 16], the
// result lane l holds D[4 (l / 16) + v][l % 16].
//
// Edges.  x rows past M and k past K load zeros; weight rows past N and
// groups past K get scale 0 (zero weights); results past M or N are not
// stored.
#include "wq_device.h"
#include "wq_internal.h"

namespace wq {
namespace {

using namespace dev;

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float4v __attribute__((ext_vector_type(4)));

constexpr int kBM = 128;  // the tile prefill_fits counts blocks of
constexpr int kBN = 128;
constexpr int kBK = 64;
constexpr int kThreads = 256;
constexpr int kRow = kBK + 8;  // LDS row in halves: 144 bytes, which spreads rows over the banks

struct Stage {
    uint16_t a[kBM][kRow];  // x, 8-element pieces in dequantization order
    uint16_t b[kBN][kRow];  // fp16 weights (q - 8) * s, same order
};

// 8 consecutive x values (k .. k + 7) in the order a code word dequantizes:
// (0, 4), (1, 5), (2, 6), (3, 7).
__device__ __forceinline__ u32x4 to_dequant_order(const u32x4 d) {
    u32x4 r;
    r.x = __builtin_amdgcn_perm(d.z, d.x, 0x05040100u);
    r.y = __builtin_amdgcn_perm(d.z, d.x, 0x07060302u);
    r.z = __builtin_amdgcn_perm(d.w, d.y, 0x05040100u);
    r.w = __builtin_amdgcn_perm(d.w, d.y, 0x07060302u);
    return r;
}

__global__ __launch_bounds__(kThreads, 2) void prefill_kernel(const u32x4* __restrict__ packed,
                                                           const uint16_t* __restrict__ scales,
                                                           const uint16_t* __restrict__ x, uint16_t* __restrict__ y,
                                                           int m, int n, int k, int blocks_m) {
    __shared__ __align__(16) Stage st[2];
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int wm = wave >> 1, wn = wave & 1;
    const int bid = blockIdx.x;
    const int m0 = (bid % blocks_m) * kBM;
    const int n0 = (bid / blocks_m) * kBN;
    const int ng = k / kGroup;
    const int stages = (k + kBK - 1) / kBK;

    // This thread's share of a stage's global loads, in two register sets:
    // the loads of stage s + 2 are issued while stage s is multiplied and
    // stage s + 1 is written to LDS.  All loads are buffer loads whose offset
    // is set past the buffer for pieces outside the matrices (they read
    // zeros: x = 0, codes 0 with scale 0 give weight 0), so there is no
    // branch around a load and the waits stay exact.
    struct Regs {
        u32x4 a[4];
        u32x4 b;
        uint32_t s;
    };
    constexpr uint32_t kOut = kPrefillOutOffset;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(x), (short)0, (int)((uint32_t)m * (uint32_t)k * 2u), kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<u32x4*>(packed), (short)0, (int)((uint32_t)n * (uint32_t)ng * 16u), kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t sr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(scales), (short)0, (int)((uint32_t)n * (uint32_t)ng * 2u), kRawBufferFlags);
    const int bn = tid >> 1, bgrp = tid & 1;  // weight row and group (of two) of the B piece
    auto load_stage = [&](int s, Regs& R) {
        const int k0 = s * kBK;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = tid + kThreads * i;
            const int row = c >> 3, kc = c & 7;
            const int gm = m0 + row, gk = k0 + 8 * kc;
            const uint32_t off = (gm < m && gk < k) ? ((uint32_t)gm * (uint32_t)k + (uint32_t)gk) * 2u : kOut;
            R.a[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
        }
        const int gn = n0 + bn, g = 2 * s + bgrp;
        const bool ok = gn < n && g < ng;
        const uint32_t gi = (uint32_t)gn * (uint32_t)ng + (uint32_t)g;
        R.b = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(wr, ok ? gi * 16u : kOut, 0, 0));
        R.s = __builtin_amdgcn_raw_buffer_load_b16(sr, ok ? gi * 2u : kOut, 0, 0);
    };
    auto store_stage = [&](Stage& S, const Regs& R) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = tid + kThreads * i;
            const int row = c >> 3, kc = c & 7;
            *reinterpret_cast<u32x4*>(&S.a[row][8 * kc]) = to_dequant_order(R.a[i]);
        }
        const half2v sc = as_h2(R.s | (R.s << 16));
        const uint32_t w[4] = {R.b.x, R.b.y, R.b.z, R.b.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            half2v q[4];
            dequant_word(w[j], q);
            const u32x4 o = {__builtin_bit_cast(uint32_t, q[0] * sc), __builtin_bit_cast(uint32_t, q[1] * sc),
                             __builtin_bit_cast(uint32_t, q[2] * sc), __builtin_bit_cast(uint32_t, q[3] * sc)};
            *reinterpret_cast<u32x4*>(&S.b[bn][32 * bgrp + 8 * j]) = o;
        }
    };

    float4v acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = float4v{0.0f, 0.0f, 0.0f, 0.0f};

    const int r = lane & 15, c = lane >> 4;
    auto compute = [&](const Stage& S) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            half8 fa[4], fb[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                fa[i] = *reinterpret_cast<const half8*>(&S.a[64 * wm + 16 * i + r][32 * ks + 8 * c]);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                fb[j] = *reinterpret_cast<const half8*>(&S.b[64 * wn + 16 * j + r][32 * ks + 8 * c]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[i], fb[j], acc[i][j], 0, 0, 0);
        }
    };

    // Stages in pairs: LDS buffer and register set s & 1.  Loads past the
    // last stage read zeros and are never stored.
    Regs R0, R1;
    load_stage(0, R0);
    load_stage(1, R1);
    store_stage(st[0], R0);
    load_stage(2, R0);
    __syncthreads();
    for (int s = 0; s < stages; s += 2) {
        compute(st[0]);
        store_stage(st[1], R1);  // stage s + 1
        load_stage(s + 3, R1);
        __syncthreads();
        if (s + 1 == stages) break;
        compute(st[1]);
        store_stage(st[0], R0);  // stage s + 2
        load_stage(s + 4, R0);
        __syncthreads();
    }

    // D[4 c + v][r] of tile (i, j): x row 64 wm + 16 i + 4 c + v, weight row 64 wn + 16 j + r.
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int gn = n0 + 64 * wn + 16 * j + r;
            if (gn >= n) continue;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int gm = m0 + 64 * wm + 16 * i + 4 * c + v;
                if (gm < m) gbl(y)[(int64_t)gm * n + gn] = __half_as_ushort(__float2half_rn(acc[i][j][v]));
            }
        }
    }
}

}  // namespace

hipError_t launch_prefill(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y,
                          int64_t n, int64_t k, int64_t m, hipStream_t stream) {
    const int64_t blocks_m = (m + kBM - 1) / kBM;
    const int64_t blocks = blocks_m * ((n + kBN - 1) / kBN);
    hipLaunchKernelGGL(prefill_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream,
                       reinterpret_cast<const u32x4*>(packed), scales, x, y, (int)m, (int)n, (int)k, (int)blocks_m);
    return hipGetLastError();
}

}  // namespace wq
