// Host-side predicates that decide which kernel can take a shape.  Plain C++
// (no HIP types), so that host-only tests can include this header.  The
// functions are constexpr, which also makes them callable from device code.
#pragma once

#include <stdint.h>

namespace wq {

// A linear's codes (n * ng 16-byte groups) can be addressed through the
// 32-bit offsets of a buffer resource.
constexpr bool fits_rsrc(int64_t n, int64_t ng) { return n * ng * 16 <= 0xFFFFFFFFll; }

// The prefill GEMM addresses x, the codes and the scales through 32-bit
// buffer offsets and points loads of pieces outside the matrices at this
// offset, which must lie past every buffer's end so that they read zeros.
constexpr uint32_t kPrefillOutOffset = 0xFFFFFFF0u;

// The prefill GEMM takes (n, k, m) when its sizes and block count fit int32
// and x (m * k * 2 bytes) and the codes (n * k / 2 bytes) stay at or below
// kPrefillOutOffset bytes; otherwise wq_gemv runs the generic kernel.
constexpr bool prefill_fits(int64_t n, int64_t k, int64_t m) {
    return n > 0 && k > 0 && m > 0 && n <= INT32_MAX && k <= INT32_MAX && m <= INT32_MAX &&
           ((m + 127) / 128) * ((n + 127) / 128) <= INT32_MAX && m * k * 2 <= (int64_t)kPrefillOutOffset &&
           n * (k / 32) * 16 <= (int64_t)kPrefillOutOffset;
}

}  // namespace wq
