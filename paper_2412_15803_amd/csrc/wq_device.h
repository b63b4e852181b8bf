// Device-side building blocks shared by the GEMV and decode-step kernels
// (gfx950, wave64).
//
// Weight format (the paper's ahead-of-time 4-bit conversion, Sec. 2.3 and
// Table 1): packed [N][K/8] uint32, element 8j+i of a row in bits [4i, 4i+4)
// of word j; fp16 scales [N][K/32].  One 16-byte load of packed data is one
// 32-element group of one row.
//
// Numerics: codes become the exact fp16 integers q - 8; products with fp16 x
// are exact inside v_dot2 (fp16 x fp16 fits in fp32) and accumulate in fp32;
// the group scale is applied once per group in fp32; each output is rounded
// once to fp16.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wq {
namespace dev {

typedef _Float16 half2v __attribute__((ext_vector_type(2)));

constexpr int kGroup = 32;
constexpr int kWave = 64;

__device__ __forceinline__ half2v as_h2(uint32_t v) { return __builtin_bit_cast(half2v, v); }

// x for one group (32 fp16) as 16 half2 pairs, per word c ordered
// (x[8c+0], x[8c+4]), (x[8c+1], x[8c+5]), (x[8c+2], x[8c+6]), (x[8c+3], x[8c+7]):
// the nibble pairs that one mask picks out of a word.  Masking a word with
// 0x000F000F gives codes (0, 4) in its two halves and 0x00F000F0 gives
// 16 * codes (1, 5); the same on the word shifted right by 8 gives (2, 6)
// and 16 * (3, 7).  OR-ing 0x6400 into a half makes the fp16 value 1024 + v,
// and (1024 + q) - 1032 = q - 8 = (1024 + 16 q) / 16 - 72 exactly.
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

// ------------------------------------------------------- batch-1 row steps
//
// A "step" is U consecutive rows of one linear.  Lane l owns groups
// l, l + 64, ..., l + 64 (GPL - 1) of every row, so each wave-wide 16-byte
// load covers 1 KiB of one row contiguously.  A step holds U * GPL <= 8
// loads per lane.
template <int GPL>
struct StepShape {
    static constexpr int U = GPL >= 8 ? 1 : 8 / GPL;  // rows per step
};

struct StepBuf {
    uint4 w[8];
    uint32_t s[8];
};

// x groups of this lane for one linear.  Lanes whose group index runs past
// the row get zeros and a disabled flag.
template <int GPL, int MAXG>
__device__ __forceinline__ void load_x_lane(const uint16_t* __restrict__ x, int ng, int lane,
                                            half2v (&xr)[MAXG][16], bool (&act)[MAXG]) {
#pragma unroll
    for (int j = 0; j < GPL; ++j) {
        const int g = lane + kWave * j;
        act[j] = g < ng;
        const int gc = act[j] ? g : ng - 1;
        load_x_group(x + (int64_t)gc * kGroup, xr[j]);
        if (!act[j]) {
#pragma unroll
            for (int p = 0; p < 16; ++p) xr[j][p] = half2v{(_Float16)0.0f, (_Float16)0.0f};
        }
    }
}

// Issue the loads of rows [row0, row0 + U) (clamped to last_row, so every
// lane always loads a valid address and no branch is needed).
template <int GPL>
__device__ __forceinline__ void issue_step(StepBuf& b, const uint4* packed,
                                           const uint16_t* scales, int64_t row0,
                                           int64_t last_row, int ng, int lane) {
    constexpr int U = StepShape<GPL>::U;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t r = min(row0 + u, last_row);
#pragma unroll
        for (int j = 0; j < GPL; ++j) {
            const int g = min(lane + kWave * j, ng - 1);
            const int64_t idx = r * ng + g;
            b.w[u * GPL + j] = packed[idx];
            b.s[u * GPL + j] = scales[idx];
        }
    }
    // Keep this step's loads ahead of anything issued later: the load counter
    // retires in issue order, so a later step's loads must not be scheduled
    // in between, or waiting for this step would wait for those too.  The asm
    // statement stops IR-level motion (the weight pointers are deliberately
    // not __restrict__, so it binds them), the builtin the machine scheduler.
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// Dot products, wave reduction and fp16 store of the rows of one step;
// only rows below row0 + nrows are written.
template <int GPL, int MAXG>
__device__ __forceinline__ void compute_step(const StepBuf& b, const half2v (&xr)[MAXG][16],
                                             const bool (&act)[MAXG], uint16_t* __restrict__ y,
                                             int64_t row0, int nrows, int lane) {
    constexpr int U = StepShape<GPL>::U;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        float acc = 0.0f;
#pragma unroll
        for (int j = 0; j < GPL; ++j) {
            const float s = act[j] ? __half2float(__ushort_as_half((uint16_t)b.s[u * GPL + j])) : 0.0f;
            acc = fmaf(s, dot_group(b.w[u * GPL + j], xr[j]), acc);
        }
        const float tot = wave_sum_to_last_lane(acc);
        if (lane == kWave - 1 && u < nrows) y[row0 + u] = __half_as_ushort(__float2half_rn(tot));
    }
}

}  // namespace dev
}  // namespace wq
