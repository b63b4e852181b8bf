// Internal launch interface between the C-ABI layer (wq_api.hip) and the
// kernels (wq_kernels.hip).  Arguments are already validated by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wq {

// Quantize + pack: one thread per (row, group).
hipError_t launch_pack(const float* w, uint32_t* packed, uint16_t* scales,
                       int64_t n, int64_t k, hipStream_t stream);

// y[M][N] = x[M][K] * dequant(W)^T, picking the kernel for (M, K).
hipError_t launch_gemv(const uint32_t* packed, const uint16_t* scales,
                       const uint16_t* x, uint16_t* y,
                       int64_t n, int64_t k, int64_t m, hipStream_t stream);

}  // namespace wq
