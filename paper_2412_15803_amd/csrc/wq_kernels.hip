// HIP kernels (gfx950, wave64) for 4-bit group-quantized decode linears.
//
// Format (the 4-bit weight conversion of the paper, Sec. 2.3, Table 1):
// W [N][K] fp32 -> packed [N][K/8] uint32 (element 8j+i of a row in bits
// [4i, 4i+4) of word j) + scales [N][K/32] fp16, groups of 32 along K.
// One 16-byte load of packed data is exactly one group of one row.
//
// GEMV numerics: every code is turned into the exact fp16 integer q - 8, and
// products with fp16 x are formed exactly inside v_dot2 (fp16 x fp16 fits in
// fp32) and accumulated in fp32; the fp16 group scale is applied once per
// group in fp32 and the row sum is rounded once to fp16.
#include "wq_internal.h"

#include <hip/hip_fp16.h>

namespace wq {
namespace {

typedef _Float16 half2v __attribute__((ext_vector_type(2)));

constexpr int kGroup = 32;
constexpr int kWave = 64;
constexpr int kBlock = 256;               // 4 waves per workgroup
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kTargetWaves = 256 * 8;     // 256 CUs x 8 resident waves

__device__ __forceinline__ half2v as_h2(uint32_t v) { return __builtin_bit_cast(half2v, v); }

// --------------------------------------------------------------- quantize
//
// One thread per (row, group).  Bit-exact: IEEE fp32 division (__fdiv_rn),
// round-to-nearest-even fp32->fp16 with subnormals, rintf (ties to even).
__global__ __launch_bounds__(kBlock) void pack_kernel(const float* __restrict__ w,
                                                      uint32_t* __restrict__ packed,
                                                      uint16_t* __restrict__ scales,
                                                      int64_t n, int64_t k) {
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

// ------------------------------------------------------------ dequant-dot
//
// x for one group (32 fp16) is kept as 16 half2 pairs ordered per word c as
// (x[8c+0], x[8c+4]), (x[8c+1], x[8c+5]), (x[8c+2], x[8c+6]), (x[8c+3], x[8c+7]),
// matching the nibble pairs that one AND picks out of a word: masking a word
// with 0x000F000F gives codes (0, 4) in the two halves, 0x00F000F0 gives
// 16 * codes (1, 5); the same on the word shifted right by 8 gives (2, 6) and
// 16 * (3, 7).  OR-ing 0x6400 into a half makes the fp16 value 1024 + v, and
// (1024 + q) - 1032 or (1024 + 16q) / 16 - 72 is exactly q - 8.
__device__ __forceinline__ void load_x_group(const uint16_t* __restrict__ xg, half2v out[16]) {
    const uint4* src = reinterpret_cast<const uint4*>(xg);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const uint4 d = src[c];
        out[4 * c + 0] = as_h2((d.x & 0xFFFFu) | (d.z << 16));
        out[4 * c + 1] = as_h2((d.x >> 16) | (d.z & 0xFFFF0000u));
        out[4 * c + 2] = as_h2((d.y & 0xFFFFu) | (d.w << 16));
        out[4 * c + 3] = as_h2((d.y >> 16) | (d.w & 0xFFFF0000u));
    }
}

__device__ __forceinline__ float dot_word(uint32_t w, const half2v* xp, float acc) {
    const half2v k1032 = {(_Float16)1032.0f, (_Float16)1032.0f};
    const half2v k1_16 = {(_Float16)0.0625f, (_Float16)0.0625f};
    const half2v km72 = {(_Float16)-72.0f, (_Float16)-72.0f};
    const uint32_t w8 = w >> 8;
    const half2v q04 = as_h2((w & 0x000F000Fu) | 0x64006400u) - k1032;
    const half2v q15 = as_h2((w & 0x00F000F0u) | 0x64006400u) * k1_16 + km72;
    const half2v q26 = as_h2((w8 & 0x000F000Fu) | 0x64006400u) - k1032;
    const half2v q37 = as_h2((w8 & 0x00F000F0u) | 0x64006400u) * k1_16 + km72;
    acc = __builtin_amdgcn_fdot2(q04, xp[0], acc, false);
    acc = __builtin_amdgcn_fdot2(q15, xp[1], acc, false);
    acc = __builtin_amdgcn_fdot2(q26, xp[2], acc, false);
    acc = __builtin_amdgcn_fdot2(q37, xp[3], acc, false);
    return acc;
}

// sum_{k in group} (q_k - 8) * x_k for one 16-byte group of codes.
__device__ __forceinline__ float dot_group(const uint4 wv, const half2v xg[16]) {
    float a0 = dot_word(wv.x, xg + 0, 0.0f);
    float a1 = dot_word(wv.y, xg + 4, 0.0f);
    a0 = dot_word(wv.z, xg + 8, a0);
    a1 = dot_word(wv.w, xg + 12, a1);
    return a0 + a1;
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_add(float v) {
    const int t = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROW_MASK, 0xF, false);
    return v + __builtin_bit_cast(float, t);
}

// Sum over the 64 lanes of a wave; the total lands in lane 63.
__device__ __forceinline__ float wave_sum_to_last_lane(float v) {
    v = dpp_add<0xB1, 0xF>(v);   // quad_perm [1,0,3,2]
    v = dpp_add<0x4E, 0xF>(v);   // quad_perm [2,3,0,1]
    v = dpp_add<0x141, 0xF>(v);  // row_half_mirror: 8-lane sums
    v = dpp_add<0x140, 0xF>(v);  // row_mirror: 16-lane sums
    v = dpp_add<0x142, 0xA>(v);  // row_bcast:15 into rows 1, 3
    v = dpp_add<0x143, 0xC>(v);  // row_bcast:31 into rows 2, 3
    return v;
}

// ------------------------------------------------------------ batch-1 GEMV
//
// Each wave owns a contiguous block of rows.  Lane l handles groups
// l, l + 64, ..., so one wave-wide 16-byte load reads 1 KiB of one row
// contiguously; the lane's x groups stay in registers for all its rows.
// U rows are processed per step, with the next step's loads issued before
// the current step's arithmetic.
template <int GPL, int U>
__global__ __launch_bounds__(kBlock) void gemv_m1_kernel(const uint4* __restrict__ packed,
                                                         const uint16_t* __restrict__ scales,
                                                         const uint16_t* __restrict__ x,
                                                         uint16_t* __restrict__ y,
                                                         int64_t n, int ng, int64_t rows_per_wave) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t wave = (int64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave;
    const int64_t row_begin = wave * rows_per_wave;
    if (row_begin >= n) return;
    const int64_t row_end = min(n, row_begin + rows_per_wave);

    half2v xr[GPL][16];
    bool act[GPL];
#pragma unroll
    for (int j = 0; j < GPL; ++j) {
        const int g = lane + kWave * j;
        act[j] = g < ng;
        if (act[j]) {
            load_x_group(x + (int64_t)g * kGroup, xr[j]);
        } else {
#pragma unroll
            for (int p = 0; p < 16; ++p) xr[j][p] = half2v{(_Float16)0.0f, (_Float16)0.0f};
        }
    }

    uint4 wcur[U][GPL];
    uint16_t scur[U][GPL];
    auto load_step = [&](int64_t r0, uint4 (&wv)[U][GPL], uint16_t (&sv)[U][GPL]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t r = r0 + u;
#pragma unroll
            for (int j = 0; j < GPL; ++j) {
                const int g = lane + kWave * j;
                if (act[j] && r < row_end) {
                    const int64_t idx = r * ng + g;
                    wv[u][j] = packed[idx];
                    sv[u][j] = scales[idx];
                } else {
                    wv[u][j] = make_uint4(0x88888888u, 0x88888888u, 0x88888888u, 0x88888888u);
                    sv[u][j] = 0;
                }
            }
        }
    };

    load_step(row_begin, wcur, scur);
    for (int64_t r0 = row_begin; r0 < row_end; r0 += U) {
        uint4 wnext[U][GPL];
        uint16_t snext[U][GPL];
        if (r0 + U < row_end) load_step(r0 + U, wnext, snext);

        float acc[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            acc[u] = 0.0f;
#pragma unroll
            for (int j = 0; j < GPL; ++j) {
                const float s = __half2float(__ushort_as_half(scur[u][j]));
                acc[u] = fmaf(s, dot_group(wcur[u][j], xr[j]), acc[u]);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const float tot = wave_sum_to_last_lane(acc[u]);
            if (lane == kWave - 1 && r0 + u < row_end) y[r0 + u] = __half_as_ushort(__float2half_rn(tot));
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int j = 0; j < GPL; ++j) {
                wcur[u][j] = wnext[u][j];
                scur[u][j] = snext[u][j];
            }
    }
}

// ------------------------------------------------------- generic GEMV (any M)
//
// One wave per (row, chunk of up to MC batch rows); lanes stride over the
// row's groups and read x straight from global memory.  Used for shapes the
// tuned kernels do not cover (M > 1 for now, K > 16384 at M = 1).
template <int MC>
__global__ __launch_bounds__(kBlock) void gemv_generic_kernel(const uint4* __restrict__ packed,
                                                              const uint16_t* __restrict__ scales,
                                                              const uint16_t* __restrict__ x,
                                                              uint16_t* __restrict__ y,
                                                              int64_t n, int64_t ng, int64_t m,
                                                              int64_t mchunks) {
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t total = n * mchunks;
    const int64_t wave_stride = (int64_t)gridDim.x * kWavesPerBlock;
    for (int64_t wave = (int64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave; wave < total;
         wave += wave_stride) {
    const int64_t row = wave / mchunks;
    const int64_t m0 = (wave - row * mchunks) * MC;
    const int mcount = (int)min((int64_t)MC, m - m0);
    const int64_t k = ng * kGroup;

    float acc[MC];
#pragma unroll
    for (int i = 0; i < MC; ++i) acc[i] = 0.0f;
    for (int64_t g = lane; g < ng; g += kWave) {
        const uint4 wv = packed[row * ng + g];
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
        const float tot = wave_sum_to_last_lane(acc[i]);
        if (lane == kWave - 1 && i < mcount) y[(m0 + i) * n + row] = __half_as_ushort(__float2half_rn(tot));
    }
    }
}

template <int GPL, int U>
hipError_t launch_m1(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y,
                     int64_t n, int64_t ng, hipStream_t stream) {
    const int64_t steps = (n + U - 1) / U;
    const int64_t steps_per_wave = (steps + kTargetWaves - 1) / kTargetWaves;
    const int64_t rows_per_wave = steps_per_wave * U;
    const int64_t waves = (n + rows_per_wave - 1) / rows_per_wave;
    const int64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
    hipLaunchKernelGGL((gemv_m1_kernel<GPL, U>), dim3((unsigned)blocks), dim3(kBlock), 0, stream,
                       reinterpret_cast<const uint4*>(packed), scales, x, y, n, (int)ng, rows_per_wave);
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
    if (m == 1) {
        const int64_t gpl = (ng + kWave - 1) / kWave;
        switch (gpl) {
            case 1: return launch_m1<1, 8>(packed, scales, x, y, n, ng, stream);
            case 2: return launch_m1<2, 4>(packed, scales, x, y, n, ng, stream);
            case 3: return launch_m1<3, 2>(packed, scales, x, y, n, ng, stream);
            case 4: return launch_m1<4, 2>(packed, scales, x, y, n, ng, stream);
            case 5: return launch_m1<5, 1>(packed, scales, x, y, n, ng, stream);
            case 6: return launch_m1<6, 1>(packed, scales, x, y, n, ng, stream);
            case 7: return launch_m1<7, 1>(packed, scales, x, y, n, ng, stream);
            case 8: return launch_m1<8, 1>(packed, scales, x, y, n, ng, stream);
            default: break;
        }
    }
    constexpr int MC = 4;
    const int64_t mchunks = (m + MC - 1) / MC;
    const int64_t waves = n * mchunks;
    const int64_t blocks = min((waves + kWavesPerBlock - 1) / kWavesPerBlock, (int64_t)1 << 20);
    hipLaunchKernelGGL((gemv_generic_kernel<MC>), dim3((unsigned)blocks), dim3(kBlock), 0, stream,
                       reinterpret_cast<const uint4*>(packed), scales, x, y, n, ng, m, mchunks);
    return hipGetLastError();
}

}  // namespace wq
