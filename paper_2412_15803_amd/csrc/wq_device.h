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

#include "wq_limits.h"

namespace wq {
namespace dev {

typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // one 16-byte load

constexpr int kGroup = 32;
constexpr int kWave = 64;

__device__ __forceinline__ half2v as_h2(uint32_t v) { return __builtin_bit_cast(half2v, v); }

// Global-address-space views of device pointers.  Pointers read from a table
// are generic to the compiler, which would otherwise emit FLAT accesses; those
// count on the scalar-memory counter too, so every wait for a table read
// would also wait for all weight loads in flight.
#define WQ_GLOBAL __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ const WQ_GLOBAL T* gbl(const T* p) {
    return (const WQ_GLOBAL T*)p;
}
template <typename T>
__device__ __forceinline__ WQ_GLOBAL T* gbl(T* p) {
    return (WQ_GLOBAL T*)p;
}

// x for one group (32 fp16) as 16 half2 pairs, per word c ordered
// (x[8c+0], x[8c+4]), (x[8c+1], x[8c+5]), (x[8c+2], x[8c+6]), (x[8c+3], x[8c+7]):
// the nibble pairs that one mask picks out of a word.  Masking a word with
// 0x000F000F gives codes (0, 4) in its two halves and 0x00F000F0 gives
// 16 * codes (1, 5); the same on the word shifted right by 8 gives (2, 6)
// and 16 * (3, 7).  OR-ing 0x6400 into a half makes the fp16 value 1024 + v,
// and (1024 + q) - 1032 = q - 8 = (1024 + 16 q) / 16 - 72 exactly.
__device__ __forceinline__ void load_x_group(const uint16_t* __restrict__ xg, half2v out[16]) {
    const WQ_GLOBAL u32x4* src = gbl(reinterpret_cast<const u32x4*>(xg));
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const u32x4 d = src[c];
        out[4 * c + 0] = as_h2((d.x & 0xFFFFu) | (d.z << 16));
        out[4 * c + 1] = as_h2((d.x >> 16) | (d.z & 0xFFFF0000u));
        out[4 * c + 2] = as_h2((d.y & 0xFFFFu) | (d.w << 16));
        out[4 * c + 3] = as_h2((d.y >> 16) | (d.w & 0xFFFF0000u));
    }
}

// (w & mask) | magic in one VALU op.  The constants live in registers
// (loop-invariant), which the three-operand form needs on this target.
__device__ __forceinline__ uint32_t and_or(uint32_t w, uint32_t mask, uint32_t magic) {
    uint32_t r;
    asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(w), "v"(mask), "v"(magic));
    return r;
}

// The eight codes of one word as exact fp16 (q - 8) pairs, ordered
// (0, 4), (1, 5), (2, 6), (3, 7).
__device__ __forceinline__ void dequant_word(uint32_t w, half2v (&q)[4]) {
    const half2v k1032 = {(_Float16)1032.0f, (_Float16)1032.0f};
    const half2v k1_16 = {(_Float16)0.0625f, (_Float16)0.0625f};
    const half2v km72 = {(_Float16)-72.0f, (_Float16)-72.0f};
    const uint32_t w8 = w >> 8;
    q[0] = as_h2(and_or(w, 0x000F000Fu, 0x64006400u)) - k1032;
    q[1] = as_h2(and_or(w, 0x00F000F0u, 0x64006400u)) * k1_16 + km72;
    q[2] = as_h2(and_or(w8, 0x000F000Fu, 0x64006400u)) - k1032;
    q[3] = as_h2(and_or(w8, 0x00F000F0u, 0x64006400u)) * k1_16 + km72;
}

// a.lo b.lo + a.hi b.hi in fp32, starting a chain: the three-operand form
// with an inline zero, where the compiler would otherwise copy a zero into
// the accumulator and use the two-operand form.
__device__ __forceinline__ float dot2_first(half2v a, half2v b) {
    float r;
    asm("v_dot2_f32_f16 %0, %1, %2, 0" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

__device__ __forceinline__ float dot_word(uint32_t w, const half2v* xp, float acc) {
    half2v q[4];
    dequant_word(w, q);
    acc = __builtin_amdgcn_fdot2(q[0], xp[0], acc, false);
    acc = __builtin_amdgcn_fdot2(q[1], xp[1], acc, false);
    acc = __builtin_amdgcn_fdot2(q[2], xp[2], acc, false);
    acc = __builtin_amdgcn_fdot2(q[3], xp[3], acc, false);
    return acc;
}

// sum_{k in group} (q_k - 8) * x_k for one 16-byte group of codes: one
// chain of 16 dot products, words in order.
__device__ __forceinline__ float dot_group(const u32x4 wv, const half2v xg[16]) {
    half2v q[4];
    dequant_word(wv.x, q);
    float a = dot2_first(q[0], xg[0]);
    a = __builtin_amdgcn_fdot2(q[1], xg[1], a, false);
    a = __builtin_amdgcn_fdot2(q[2], xg[2], a, false);
    a = __builtin_amdgcn_fdot2(q[3], xg[3], a, false);
    a = dot_word(wv.y, xg + 4, a);
    a = dot_word(wv.z, xg + 8, a);
    return dot_word(wv.w, xg + 12, a);
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_add(float v) {
    const int t = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, ROW_MASK, 0xF, false);
    return v + __builtin_bit_cast(float, t);
}

// Sum over each aligned segment of LPR lanes (16, 32 or 64); the segment's
// total lands in its last lane.
template <int LPR>
__device__ __forceinline__ float segment_sum(float v) {
    v = dpp_add<0xB1, 0xF>(v);   // quad_perm [1,0,3,2]
    v = dpp_add<0x4E, 0xF>(v);   // quad_perm [2,3,0,1]
    v = dpp_add<0x141, 0xF>(v);  // row_half_mirror: 8-lane sums
    v = dpp_add<0x140, 0xF>(v);  // row_mirror: 16-lane sums in every lane of a row
    if constexpr (LPR >= 32) v = dpp_add<0x142, 0xA>(v);  // row_bcast:15 into rows 1, 3
    if constexpr (LPR >= 64) v = dpp_add<0x143, 0xC>(v);  // row_bcast:31 into rows 2, 3
    return v;
}

// ------------------------------------------------------- batch-1 row steps
//
// A wave is split into 64/LPR slots of LPR lanes; each slot works on its own
// row.  Lane `sub` of a slot owns groups sub, sub + LPR, ...,
// sub + LPR (GPL - 1) of that row, so one wave-wide 16-byte load reads LPR x
// 16 contiguous bytes of each slot's row.  LPR is chosen per shape so that
// LPR * GPL covers the row's groups with no idle lanes where possible.
//
// A "step" is U rows per slot (U * 64/LPR rows per wave) and U * GPL loads
// per lane; slot s takes rows row0 + s*U .. row0 + s*U + U - 1.
// Loads of 16 bytes per lane in one step (rows per slot = this / GPL, at
// least one), by default.  Six measured best on the 8B-class decode step
// (whose K=4096 linears then take three rows per slot, in the step kernel's
// wide variant); the narrow variant and the single-linear kernels take
// fewer.
#ifndef WQ_STEP_LOADS
#define WQ_STEP_LOADS 6
#endif

__host__ __device__ constexpr int step_rows_per_slot(int gpl, int loads = WQ_STEP_LOADS) {
    return gpl >= loads ? 1 : loads / gpl;
}

// Loads per step of the batch-1 step kernel's narrow variant (up to four
// groups of x per lane) and its wide variant; its plans number steps with
// the same counts.
#ifndef WQ_GROUPED_LOADS4
#define WQ_GROUPED_LOADS4 4
#endif
#ifndef WQ_GROUPED_LOADS8
#define WQ_GROUPED_LOADS8 WQ_STEP_LOADS
#endif
__host__ __device__ constexpr int grouped_step_loads(int max_gpl) {
    return max_gpl <= 4 ? WQ_GROUPED_LOADS4 : WQ_GROUPED_LOADS8;
}

// A kernel may take steps of fewer loads (LOADS, at most 8) than the decode
// step's.
template <int LPR, int GPL, int LOADS = WQ_STEP_LOADS>
struct StepShape {
    static constexpr int SLOTS = kWave / LPR;
    static constexpr int U = step_rows_per_slot(GPL, LOADS);  // rows per slot
    static constexpr int ROWS = U * SLOTS;                    // rows per step
};

// One step's loads: per row and group, the 16-byte group of codes and its
// 2-byte scale.
struct StepBuf {
    u32x4 w[WQ_STEP_LOADS > 8 ? WQ_STEP_LOADS : 8];
    uint32_t s[WQ_STEP_LOADS > 8 ? WQ_STEP_LOADS : 8];
};

// Orders one wave's LDS accesses across its lanes: a wave's LDS operations
// execute in issue order, so it is enough to keep the compiler from moving
// them across this point.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// x groups of this lane, in two halves so that other loads can be issued
// between them: load_x_raw issues the loads of every group (one round trip
// for all), pair_x rearranges them to the dequantized codes' pairing (lanes
// whose group index runs past the row get zeros), which waits for them.
template <int LPR, int GPL, int MAXG>
__device__ __forceinline__ void load_x_raw(const uint16_t* x, int ng, int lane, u32x4 (&raw)[MAXG][4]) {
    const int sub = lane & (LPR - 1);
#pragma unroll
    for (int j = 0; j < GPL; ++j) {
        const WQ_GLOBAL u32x4* src = gbl(reinterpret_cast<const u32x4*>(x + (int64_t)min(sub + LPR * j, ng - 1) * kGroup));
#pragma unroll
        for (int c = 0; c < 4; ++c) raw[j][c] = src[c];
    }
}

template <int LPR, int GPL, int MAXG>
__device__ __forceinline__ void pair_x(const u32x4 (&raw)[MAXG][4], int ng, int lane, half2v (&xr)[MAXG][16]) {
    const int sub = lane & (LPR - 1);
#pragma unroll
    for (int j = 0; j < GPL; ++j) {
        const bool act = sub + LPR * j < ng;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const u32x4 d = raw[j][c];
            xr[j][4 * c + 0] = as_h2(act ? (d.x & 0xFFFFu) | (d.z << 16) : 0u);
            xr[j][4 * c + 1] = as_h2(act ? (d.x >> 16) | (d.z & 0xFFFF0000u) : 0u);
            xr[j][4 * c + 2] = as_h2(act ? (d.y & 0xFFFFu) | (d.w << 16) : 0u);
            xr[j][4 * c + 3] = as_h2(act ? (d.y >> 16) | (d.w & 0xFFFF0000u) : 0u);
        }
    }
}

// Keeps the loads issued so far ahead of any issued later: the compiler
// may otherwise schedule later loads first (the load counter retires in
// issue order, so a wait for the earlier loads would then wait for those).
__device__ __forceinline__ void load_order_fence() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// Both halves at once, when nothing is to be issued in between.
template <int LPR, int GPL, int MAXG>
__device__ __forceinline__ void load_x_lane(const uint16_t* x, int ng, int lane, half2v (&xr)[MAXG][16]) {
    u32x4 raw[MAXG][4];
    load_x_raw<LPR, GPL, MAXG>(x, ng, lane, raw);
    pair_x<LPR, GPL, MAXG>(raw, ng, lane, xr);
}

// Buffer resources over one linear's codes and scales.  A load's byte offset
// is this lane's offset within a step (the same vector register for every
// step) plus a wave-uniform scalar offset for the step, row and group, so
// issuing a step costs no vector address arithmetic.  The range check covers
// the sum (checked on the device: a read whose scalar offset alone passes the
// end returns zeros), so the rows past N in a linear's last step read zeros
// and nothing out of bounds.  Offsets are 32-bit: a linear is read this way
// only when its codes fit in 4 GiB (the launchers check).
struct LinearRsrc {
    __amdgpu_buffer_rsrc_t w;  // codes, n * ng * 16 bytes
    __amdgpu_buffer_rsrc_t s;  // scales, n * ng * 2 bytes
};

constexpr int kRawBufferFlags = 0x00020000;  // word 3 of a raw (unswizzled) gfx9 buffer resource

// Cache policy of a buffer load: the default, or non-temporal (the lines are
// marked as streamed and go first, so the weight stream does not push x and
// the plan out of L2).  The whole-step kernel loads its weights
// non-temporally: measured 4-6% faster on the 3B- and 8B-class steps.  Not
// the single-linear kernels (the 8B down projection alone got slower), nor
// the matrix-core kernel, whose loads read half an L2 line each and lose the
// other half before the next item reads it.
constexpr int kCpolDefault = 0;
constexpr int kCpolNonTemporal = 2;

// From the two base pointers and the scales' size in bytes (n * ng * 2; the
// codes take eight times that).
__device__ __forceinline__ LinearRsrc make_rsrc(const void* packed, const uint16_t* scales, uint32_t scale_bytes) {
    LinearRsrc r;
    r.w = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(packed), (short)0, (int)(scale_bytes * 8u),
                                            kRawBufferFlags);
    r.s = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(scales), (short)0, (int)scale_bytes,
                                            kRawBufferFlags);
    return r;
}

// Issue the loads of rows [row0, row0 + ROWS) of a linear with ng groups per
// row.  Lanes whose group index runs past the row read the next row's codes
// (or zeros at the end); their x is zero, so those codes add nothing.
template <int LPR, int GPL, int CPOL = kCpolDefault, int LOADS = WQ_STEP_LOADS>
__device__ __forceinline__ void issue_step(StepBuf& b, const LinearRsrc& r, int64_t row0, int ng, int lane) {
    using S = StepShape<LPR, GPL, LOADS>;
    const int slot = lane / LPR;
    const int sub = lane & (LPR - 1);
    // This lane's group index relative to the step's first group.
    const uint32_t lg = (uint32_t)(slot * S::U * ng + sub);
    const uint32_t g0 = (uint32_t)(row0 * ng);  // wave-uniform
#pragma unroll
    for (int u = 0; u < S::U; ++u) {
#pragma unroll
        for (int j = 0; j < GPL; ++j) {
            const uint32_t go = g0 + (uint32_t)(u * ng + LPR * j);  // wave-uniform
            b.w[u * GPL + j] =
                __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r.w, lg * 16, go * 16, CPOL));
            b.s[u * GPL + j] = __builtin_amdgcn_raw_buffer_load_b16(r.s, lg * 2, go * 2, CPOL);
        }
    }
    // Keep this step's loads ahead of anything issued later: the load counter
    // retires in issue order, so a later step's loads must not be scheduled
    // in between, or waiting for this step would wait for those too.
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// Whether a linear's codes can be addressed through 32-bit buffer offsets.
using wq::fits_rsrc;

// Dot products, segment reduction and fp16 rounding of one step; the rows
// below nrows are staged in this wave's LDS slice at ylds[yrel + row], to be
// written out by flush_y.  (Global stores inside the loop would share the
// load counter with the weight loads in flight, and every later wait for a
// step's loads would then also wait for those stores.)  Lanes past the
// row's groups hold zero x, so their (clamped, finite) codes contribute
// nothing.
template <int LPR, int GPL, int MAXG, int LOADS = WQ_STEP_LOADS>
__device__ __forceinline__ void compute_step(const StepBuf& b, const half2v (&xr)[MAXG][16], int nrows,
                                             uint16_t* ylds, int yrel, int lane) {
    using S = StepShape<LPR, GPL, LOADS>;
    const int slot = lane / LPR;
    const int sub = lane & (LPR - 1);
#pragma unroll
    for (int u = 0; u < S::U; ++u) {
        float acc = 0.0f;
#pragma unroll
        for (int j = 0; j < GPL; ++j) {
            const float s = __half2float(__ushort_as_half((uint16_t)b.s[u * GPL + j]));
            acc = fmaf(s, dot_group(b.w[u * GPL + j], xr[j]), acc);
        }
        const float tot = segment_sum<LPR>(acc);
        const int rr = slot * S::U + u;
        if (sub == LPR - 1 && rr < nrows) ylds[yrel + rr] = __half_as_ushort(__float2half_rn(tot));
    }
}

// Rows of y a wave stages in LDS before writing them out (2 KiB per wave).
// Launches and plans cap a wave's rows at the largest multiple of its rows
// per step that fits.
constexpr int kYRows = 1024;

// Write the `count` staged rows ylds[0, count) to y[row0, row0 + count),
// 64 consecutive rows per store instruction.
__device__ __forceinline__ void flush_y(uint16_t* y, int64_t row0, const uint16_t* ylds, int count, int lane) {
    wave_lds_sync();
    WQ_GLOBAL uint16_t* dst = gbl(y) + row0;
    for (int i = lane; i < count; i += kWave) dst[i] = ylds[i];
    wave_lds_sync();  // stores have read the slice before it is refilled
}

// Lanes per row and groups per lane for a row of ng groups (ng <= 512):
// an exact cover when one exists, else 64 lanes with the tail lanes idle.
__host__ __device__ inline void pick_shape(int ng, int& lpr, int& gpl) {
    if (ng <= 16) { lpr = 16; gpl = 1; return; }
    if (ng % 64 == 0) { lpr = 64; gpl = ng / 64; return; }
    if (ng % 32 == 0 && (ng / 32) % 2 == 1 && ng / 32 <= 7) { lpr = 32; gpl = ng / 32; return; }
    if (ng % 16 == 0 && (ng / 16) % 2 == 1 && ng / 16 <= 7) { lpr = 16; gpl = ng / 16; return; }
    lpr = 64;
    gpl = (ng + 63) / 64;
}

}  // namespace dev
}  // namespace wq
