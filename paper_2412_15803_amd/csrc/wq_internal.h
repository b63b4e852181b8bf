// Internal launch interface between the C-ABI layer (wq_api.hip) and the
// kernels (wq_kernels.hip).  Arguments are already validated by the caller.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "wq.h"
#include "wq_limits.h"

namespace wq {

// Records `message` as the calling thread's last error message (the one
// wq_last_error_message returns) and returns `st`.
wq_status record_error(wq_status st, const char* message);

// WQ_OK for hipSuccess; otherwise WQ_ERR_HIP with the runtime's message,
// recorded as the thread's last error message for entry point `fn`.
wq_status hip_error(const char* fn, hipError_t e);

// Quantize + pack: one thread per (row, group).
hipError_t launch_pack(const float* w, uint32_t* packed, uint16_t* scales,
                       int64_t n, int64_t k, hipStream_t stream);

// y[M][N] = x[M][K] * dequant(W)^T, picking the kernel for (M, K).
hipError_t launch_gemv(const uint32_t* packed, const uint16_t* scales,
                       const uint16_t* x, uint16_t* y,
                       int64_t n, int64_t k, int64_t m, hipStream_t stream);

// Smallest batch that uses the matrix cores; M = 2 runs on the vector ALUs.
// Measured on the 3B- and 8B-class decode steps: the matrix cores are faster
// from M = 3 on (3B step at M = 4: 435 against 475 us; 8B step at M = 7: 930
// against 1624 us), the vector kernel at M = 2 (395 against 479 us).
constexpr int kMatrixCoreMinM = 3;

// Largest batch of the small-batch kernels; larger ones (prompts) run the
// tiled prefill GEMM.
constexpr int kMaxSmallBatchM = 64;

// y[M][N] for M > kMaxSmallBatchM: 128 x 128 tiles on the matrix cores, for
// the shapes prefill_fits (wq_limits.h) accepts.
hipError_t launch_prefill(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y,
                          int64_t n, int64_t k, int64_t m, hipStream_t stream);

// Whether a small batch of m rows (2 <= m <= kMaxSmallBatchM) runs on the
// matrix cores: from kMatrixCoreMinM rows on.  Tuning overrides, read at
// every call (for comparing the two paths): WQ_SMALL_BATCH_VECTOR=1 sends
// every small batch to the vector kernel, WQ_MATRIX_MIN_M=n moves the
// threshold to n.
bool use_matrix_cores(int64_t m);

// y[M][N] for 2 <= M on the matrix cores, 16 batch rows per launch.
hipError_t launch_gemm_mfma(const uint32_t* packed, const uint16_t* scales, const uint16_t* x, uint16_t* y,
                            int64_t n, int64_t k, int64_t m, hipStream_t stream);

// One linear of a grouped launch as the kernel sees it (built on the host,
// uploaded once per distinct descriptor list).
struct DecodeEntry {
    const void* packed;      // [n][ng] 16-byte groups
    const uint16_t* scales;  // [n][ng]
    const uint16_t* x;       // [ng * 32]
    uint16_t* y;             // [n]
    int64_t n;
    int64_t first_step;      // first step of this linear in its class's numbering
    int64_t steps;           // steps of this linear: ceil(n / rows per step)
    int32_t ng;              // groups of 32 per row
    int32_t lpr;             // lanes per row (16, 32 or 64)
    int32_t gpl;             // groups per lane (lpr * gpl >= ng)
    int32_t pad;             // rows per wave (small-batch vector launches)
};
static_assert(sizeof(DecodeEntry) == 72, "DecodeEntry layout");

// Linears of one launch with the same step shape.  The class's steps are
// split into `blocks` equal contiguous ranges, one per workgroup, for the
// workgroups [blocks_begin, blocks_begin + blocks) of the grid.
struct DecodeClass {
    int32_t lpr, gpl;     // the class's step shape
    int32_t first;        // offset of its linears in the class list
    int32_t count;        // number of linears
    int64_t steps;        // steps over all its linears
    int32_t blocks_begin;
    int32_t blocks;
};
static_assert(sizeof(DecodeClass) == 32, "DecodeClass layout");

// One workgroup's share of its class in a grouped launch: steps [begin,
// end) of the class's numbering, and the position (in the class's list) of
// the linear that holds step `begin`.
struct DecodeBlock {
    int32_t pos;
    int32_t begin, end;
    int32_t pad;
};
static_assert(sizeof(DecodeBlock) == 16, "DecodeBlock layout");

// Device-side view of one grouped launch: the entries, the class
// descriptors, per class the indices of its linears in order, and per
// workgroup its share.
struct DecodePlan {
    const DecodeEntry* entries;
    const DecodeClass* classes;
    const int32_t* class_lin;
    const DecodeBlock* blocks;
    int32_t nclasses;
};

// Small-batch decode step: independent linears in one launch of the matrix-core
// kernel.  Entry i owns blocks [first_step, first_step + steps) of the grid,
// each block grouped_mfma_tiles() tiles of 16 rows, waves_per_block <=
// grouped_mfma_max_waves();
// batch rows [m0, m0 + m), m <= 16.
int grouped_mfma_tiles();
// Most waves a block of the matrix-core kernels has (LDS per wave).
int grouped_mfma_max_waves();
hipError_t launch_grouped_mfma(const DecodeEntry* entries, int count, int64_t blocks, int waves_per_block,
                               int64_t m0, int m, hipStream_t stream);

// Small-batch decode step below kMatrixCoreMinM rows (or any small batch when
// forced): independent linears in
// one launch of the vector kernel.  Entry i owns waves [first_step,
// first_step + steps) of the grid, `pad` rows each (a multiple of 8, at most
// 256); batch rows [m0, m0 + m), m <= 8.
hipError_t launch_grouped_mb(const DecodeEntry* entries, int count, int64_t waves, int64_t m0, int m,
                             hipStream_t stream);
// Waves to split such a launch into for m batch rows (m <= 8) on `device`:
// a few times what the device holds at once.
hipError_t mb_target_waves(int m, int device, int64_t& waves);
// Rows per wave for a linear of ng groups per row when each wave is to
// stream about `work` (row, padded group) pairs.
int mb_rows_for_work(int64_t work, int64_t ng);

// The vector small-batch kernel walks a row's groups in 32-group tiles, two
// row sets per wave, when those pad the row less than 64-group tiles do.
__host__ __device__ inline bool mb_two_sets(int64_t ng) { return (ng + 31) / 32 * 32 < (ng + 63) / 64 * 64; }
__host__ __device__ inline int64_t mb_padded_groups(int64_t ng) {
    return mb_two_sets(ng) ? (ng + 31) / 32 * 32 : (ng + 63) / 64 * 64;
}

// Largest groups-per-lane of the grouped kernel (K <= 16384).
constexpr int kDecodeMaxGpl = 8;
constexpr int kMaxClasses = 16;

// Launch the grouped batch-1 GEMV over a plan in device memory with
// `blocks` workgroups (the sum of the classes' workgroups), each one CU's
// worth of waves.
hipError_t launch_grouped_m1(const DecodePlan& plan, int max_gpl, int blocks, hipStream_t stream);

// Workgroups of the grouped kernel (for max_gpl) that the device holds at
// once: one per CU.
hipError_t grouped_capacity(int max_gpl, int device, int& blocks);

}  // namespace wq
