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

// One linear of a decode step as the persistent decode kernel sees it
// (built on the host, uploaded once per distinct descriptor list).
struct DecodeEntry {
    const void* packed;      // [n][ng] 16-byte groups
    const uint16_t* scales;  // [n][ng]
    const uint16_t* x;       // [ng * 32]
    uint16_t* y;             // [n]
    int64_t n;
    int32_t ng;              // groups of 32 per row
    int32_t gpl;             // groups per lane: ceil(ng / 64)
    int32_t tile_rows;       // rows per claimed tile (a multiple of the step height)
    int32_t tiles;           // ceil(n / tile_rows)
    int32_t first_tile;      // global index of this linear's first tile
    int32_t dep0, dep1;      // linears that must complete before this one reads x (-1: none)
    int32_t signal;          // nonzero if a later linear waits for this one
    int32_t pad[2];
};
static_assert(sizeof(DecodeEntry) == 80, "DecodeEntry layout");

// Counter words of the decode workspace: ticket, exit count, error flag,
// reserved, then one completed-tile counter per linear.
constexpr int kSyncHeader = 4;

// Largest groups-per-lane the persistent decode kernel handles (K <= 16384).
constexpr int kDecodeMaxGpl = 8;

// Launch the persistent decode-step kernel over `count` entries already in
// device memory.  `sync` must hold kSyncHeader + count zeroed words; the
// kernel leaves them zeroed again when it finishes.
hipError_t launch_decode_m1(const DecodeEntry* table, int count, int total_tiles, int max_gpl,
                            uint32_t* sync, uint32_t spin_limit, int blocks, hipStream_t stream);

}  // namespace wq
