// Quantize+pack and single-linear GEMV kernels (gfx950, wave64).
#include "wq_device.h"
#include "wq_internal.h"

namespace wq {
namespace {

using namespace dev;

constexpr int kBlock = 256;  // 4 waves per workgroup
constexpr int kWavesPerBlock = kBlock / kWave;

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
// steps through two register buffers: compute buffer A, refill A with the
// step two ahead, compute B, refill B.  Whenever the wave waits for a buffer,
// the other buffer's loads are still in flight.  Outputs are staged in LDS
// and written once, after the last step.
template <int LPR, int GPL>
__global__ __launch_bounds__(kBlock) void gemv_m1_kernel(const u32x4* packed, const uint16_t* scales,
                                                         const uint16_t* __restrict__ x,
                                                         uint16_t* __restrict__ y, int64_t n, int ng,
                                                         int64_t rows_per_wave) {
    constexpr int R = StepShape<LPR, GPL>::ROWS;
    const int lane = threadIdx.x & (kWave - 1);
    // Wave-uniform (the compiler cannot see that threadIdx.x / 64 is), so
    // the row bookkeeping stays in scalar registers and branches uniform.
    const int64_t wave = (int64_t)__builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock + threadIdx.x / kWave);
    const int64_t rb = wave * rows_per_wave;
    if (rb >= n) return;
    const int64_t re = min(n, rb + rows_per_wave);
    const int64_t steps = (re - rb + R - 1) / R;
    const LinearRsrc rs = make_rsrc(packed, scales, (uint32_t)(n * ng * 2));

    __shared__ __align__(16) uint16_t s_y[kWavesPerBlock][kYRows];
    uint16_t* ylds = s_y[threadIdx.x / kWave];

    half2v xr[GPL][16];
    load_x_lane<LPR, GPL, GPL>(x, ng, lane, xr);

    // The loop starts two steps early so that the first pass only issues and
    // every load comes from the same two issue sites (one register
    // assignment, no prologue copies that would force a full wait).  Every
    // issue is unconditional (past the matrix the loads read zeros), so the
    // wait counts stay exact.
    StepBuf a, b;
    for (int64_t s = -2; s < steps; s += 2) {
        const int64_t ra = rb + s * R;
        if (s >= 0) compute_step<LPR, GPL, GPL>(a, xr, (int)min((int64_t)R, re - ra), ylds, (int)(s * R), lane);
        issue_step<LPR, GPL>(a, rs, ra + 2 * R, ng, lane);
        const int64_t rbb = ra + R;
        if (s + 1 >= 0 && s + 1 < steps)
            compute_step<LPR, GPL, GPL>(b, xr, (int)min((int64_t)R, re - rbb), ylds, (int)((s + 1) * R), lane);
        issue_step<LPR, GPL>(b, rs, rbb + 2 * R, ng, lane);
    }
    flush_y(y, rb, ylds, (int)(re - rb), lane);
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

constexpr int kTargetWaves = 256 * 8;  // 256 CUs x 8 waves

template <int LPR, int GPL>
hipError_t launch_m1(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y,
                     int64_t n, int64_t ng, hipStream_t stream) {
    constexpr int R = StepShape<LPR, GPL>::ROWS;
    const int64_t steps = (n + R - 1) / R;
    // At most kYRows rows per wave (its LDS staging of y); more waves than
    // the target when the matrix is taller than that allows.
    const int64_t steps_per_wave = min((steps + kTargetWaves - 1) / kTargetWaves, (int64_t)(kYRows / R));
    const int64_t rows_per_wave = steps_per_wave * R;
    const int64_t waves = (n + rows_per_wave - 1) / rows_per_wave;
    const int64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL((gemv_m1_kernel<LPR, GPL>), dim3((unsigned)blocks), dim3(kBlock), 0, stream,
                       reinterpret_cast<const u32x4*>(packed), scales, x, y, n, (int)ng, rows_per_wave);
    return hipGetLastError();
}

}  // namespace

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
    if (m >= 2 && m <= 64 && fits_rsrc(n, ng)) return launch_gemm_mfma(packed, scales, x, y, n, k, m, stream);
    constexpr int MC = 4;
    const int64_t mchunks = (m + MC - 1) / MC;
    const int64_t waves = n * mchunks;
    const int64_t blocks = min((waves + kWavesPerBlock - 1) / kWavesPerBlock, (int64_t)1 << 20);
    hipLaunchKernelGGL((gemv_generic_kernel<MC>), dim3((unsigned)blocks), dim3(kBlock), 0, stream,
                       reinterpret_cast<const u32x4*>(packed), scales, x, y, n, ng, m, mchunks);
    return hipGetLastError();
}

}  // namespace wq
