// Persistent batch-1 decode-step kernel: every linear of a decode step in
// one launch (the per-token work of the paper's decode loop, Sec. 1 and
// Table 1; kernel fusion across operators, Sec. 2.3).
//
// Work is cut into tiles (consecutive rows of one linear).  Waves claim tiles
// in order from one atomic ticket, so a wave holding a tile of linear L knows
// that every tile of every earlier linear has already been claimed by a
// running wave.  A linear that reads another linear's output (or overwrites
// its input or output) waits, before computing, until that linear's tiles are
// all done; because claims are ordered and a wave never waits while it holds
// an uncomputed earlier step, the smallest unfinished tile can always make
// progress, whether or not all waves are resident.  Every wait is bounded: on
// overrun it sets the error word and proceeds, so the kernel always drains.
//
// Each wave streams its steps through two register buffers (compute A,
// refill A, compute B, refill B), and the weights of the next tiles --
// including tiles of the next linears -- are in flight while the current one
// is computed, so the memory pipe stays full across linear boundaries.
//
// The last wave to finish resets the counters, leaving the workspace ready
// for the next launch on the stream.
#include "wq_device.h"
#include "wq_internal.h"

namespace wq {
namespace {

using namespace dev;

constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / kWave;

struct Step {
    int lin;        // -1 when the wave has no more work
    int nrows;      // rows of this step inside its tile
    int last;       // nonzero for the last step of its tile
    int64_t row;    // first row
};

struct TileIter {
    int lin;          // linear of the current tile (scan position; tickets only grow)
    int exhausted;
    int64_t row;      // next row of the current tile
    int64_t end;      // end row of the current tile
    uint32_t pending; // pre-claimed ticket (valid in lane 0)
};

__device__ __forceinline__ uint32_t claim(uint32_t* ticket, int lane) {
    uint32_t t = 0;
    if (lane == 0) t = __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return t;
}

__device__ __forceinline__ int rows_per_step(int gpl) { return gpl >= 8 ? 1 : 8 / gpl; }

__device__ __forceinline__ Step next_step(TileIter& it, const DecodeEntry* table, int total_tiles,
                                          uint32_t* ticket, int lane) {
    Step s;
    while (it.row >= it.end) {
        if (it.exhausted) {
            s.lin = -1;
            s.nrows = 0;
            s.last = 0;
            s.row = 0;
            return s;
        }
        const uint32_t t = __builtin_amdgcn_readfirstlane(it.pending);
        if (t >= (uint32_t)total_tiles) {
            it.exhausted = 1;
            continue;
        }
        it.pending = claim(ticket, lane);  // the following tile, consumed later
        while ((int)t >= table[it.lin].first_tile + table[it.lin].tiles) ++it.lin;
        const DecodeEntry& e = table[it.lin];
        it.row = (int64_t)((int)t - e.first_tile) * e.tile_rows;
        it.end = min(e.n, it.row + e.tile_rows);
    }
    const int u = rows_per_step(table[it.lin].gpl);
    s.lin = it.lin;
    s.row = it.row;
    s.nrows = (int)min((int64_t)u, it.end - it.row);
    it.row += u;
    s.last = it.row >= it.end;
    return s;
}

template <int MAXG>
__device__ __forceinline__ void load_x_slot(const DecodeEntry& e, int lane, half2v (&xr)[MAXG][16],
                                            bool (&act)[MAXG]) {
#pragma unroll
    for (int j = 0; j < MAXG; ++j) {
        act[j] = false;
        if (j < e.gpl) {
            const int g = lane + kWave * j;
            act[j] = g < e.ng;
            load_x_group(e.x + (int64_t)min(g, e.ng - 1) * kGroup, xr[j]);
        }
    }
}

template <int MAXG>
__device__ __forceinline__ void issue_weights(StepBuf& b, const DecodeEntry& e, const Step& s, int lane) {
    const uint4* packed = reinterpret_cast<const uint4*>(e.packed);
    const int64_t last = s.row + s.nrows - 1;
    switch (e.gpl) {
        case 1: issue_step<1>(b, packed, e.scales, s.row, last, e.ng, lane); break;
        case 2: issue_step<2>(b, packed, e.scales, s.row, last, e.ng, lane); break;
        case 3: if constexpr (MAXG >= 3) issue_step<3>(b, packed, e.scales, s.row, last, e.ng, lane); break;
        case 4: if constexpr (MAXG >= 4) issue_step<4>(b, packed, e.scales, s.row, last, e.ng, lane); break;
        case 5: if constexpr (MAXG >= 5) issue_step<5>(b, packed, e.scales, s.row, last, e.ng, lane); break;
        case 6: if constexpr (MAXG >= 6) issue_step<6>(b, packed, e.scales, s.row, last, e.ng, lane); break;
        case 7: if constexpr (MAXG >= 7) issue_step<7>(b, packed, e.scales, s.row, last, e.ng, lane); break;
        default: if constexpr (MAXG >= 8) issue_step<8>(b, packed, e.scales, s.row, last, e.ng, lane); break;
    }
}

template <int MAXG>
__device__ __forceinline__ void compute_weights(const StepBuf& b, const DecodeEntry& e, const Step& s,
                                                const half2v (&xr)[MAXG][16], const bool (&act)[MAXG],
                                                int lane) {
    switch (e.gpl) {
        case 1: compute_step<1, MAXG>(b, xr, act, e.y, s.row, s.nrows, lane); break;
        case 2: compute_step<2, MAXG>(b, xr, act, e.y, s.row, s.nrows, lane); break;
        case 3: if constexpr (MAXG >= 3) compute_step<3, MAXG>(b, xr, act, e.y, s.row, s.nrows, lane); break;
        case 4: if constexpr (MAXG >= 4) compute_step<4, MAXG>(b, xr, act, e.y, s.row, s.nrows, lane); break;
        case 5: if constexpr (MAXG >= 5) compute_step<5, MAXG>(b, xr, act, e.y, s.row, s.nrows, lane); break;
        case 6: if constexpr (MAXG >= 6) compute_step<6, MAXG>(b, xr, act, e.y, s.row, s.nrows, lane); break;
        case 7: if constexpr (MAXG >= 7) compute_step<7, MAXG>(b, xr, act, e.y, s.row, s.nrows, lane); break;
        default: if constexpr (MAXG >= 8) compute_step<8, MAXG>(b, xr, act, e.y, s.row, s.nrows, lane); break;
    }
}

// Wait until linear `dep` has completed all its tiles (bounded).
__device__ __forceinline__ void wait_linear(const DecodeEntry* table, uint32_t* done, uint32_t* error, int dep,
                                            uint32_t spin_limit) {
    const uint32_t target = (uint32_t)table[dep].tiles;
    uint32_t spins = 0;
    while (__hip_atomic_load(&done[dep], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
        if (++spins > spin_limit) {
            __hip_atomic_fetch_or(error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
        }
        __builtin_amdgcn_s_sleep(2);
    }
}

// The wave's x registers and the linear they belong to.  One slot per wave:
// it is switched when the wave computes the first step of a new linear, at
// which point every earlier step of the wave has been computed.  The fresh x
// loads are then the youngest in flight, so the wave drains its pipeline once
// per linear switch; tiles are sized so that switches are rare.
template <int MAXG>
struct XSlot {
    half2v xr[MAXG][16];
    bool act[MAXG];
    int lin;
};

template <int MAXG>
__device__ __forceinline__ void issue_into(StepBuf& b, const Step& s, const DecodeEntry* table, int lane) {
    if (s.lin < 0) return;
    issue_weights<MAXG>(b, table[s.lin], s, lane);
}

template <int MAXG>
__device__ __forceinline__ void compute_from(const StepBuf& b, XSlot<MAXG>& xs, const Step& s,
                                             const DecodeEntry* table, uint32_t* done, uint32_t* error,
                                             uint32_t spin_limit, int lane) {
    if (s.lin < 0) return;
    const DecodeEntry& e = table[s.lin];
    if (xs.lin != s.lin) {
        if (e.dep0 >= 0 || e.dep1 >= 0) {
            // Every earlier step of this wave has been computed, so waiting
            // here cannot hold back a tile that the awaited linear needs.
            if (e.dep0 >= 0) wait_linear(table, done, error, e.dep0, spin_limit);
            if (e.dep1 >= 0) wait_linear(table, done, error, e.dep1, spin_limit);
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        }
        load_x_slot<MAXG>(e, lane, xs.xr, xs.act);
        xs.lin = s.lin;
    }
    compute_weights<MAXG>(b, e, s, xs.xr, xs.act, lane);
    if (s.last && e.signal && lane == kWave - 1) {
        // lane 63 wrote every y of the tile; release them with the count
        __hip_atomic_fetch_add(&done[s.lin], 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
}

template <int MAXG>
__global__ __launch_bounds__(kBlock) void decode_m1_kernel(const DecodeEntry* __restrict__ table, int count,
                                                           int total_tiles, uint32_t* sync, uint32_t spin_limit) {
    const int lane = threadIdx.x & (kWave - 1);
    uint32_t* ticket = sync;
    uint32_t* exit_count = sync + 1;
    uint32_t* error = sync + 2;
    uint32_t* done = sync + kSyncHeader;

    TileIter it;
    it.lin = 0;
    it.exhausted = 0;
    it.row = 0;
    it.end = 0;
    it.pending = claim(ticket, lane);

    StepBuf a, b;
    XSlot<MAXG> xs;
    xs.lin = -1;
    Step sa, sb;
    sa.lin = sb.lin = -1;
    sa.nrows = sb.nrows = sa.last = sb.last = 0;
    sa.row = sb.row = 0;

    // The first pass only issues; afterwards each pass computes the step a
    // buffer holds and refills that buffer with the wave's next step.
    for (;;) {
        compute_from<MAXG>(a, xs, sa, table, done, error, spin_limit, lane);
        sa = next_step(it, table, total_tiles, ticket, lane);
        issue_into<MAXG>(a, sa, table, lane);
        compute_from<MAXG>(b, xs, sb, table, done, error, spin_limit, lane);
        sb = next_step(it, table, total_tiles, ticket, lane);
        issue_into<MAXG>(b, sb, table, lane);
        if (sa.lin < 0 && sb.lin < 0) break;
    }

    // Exit: the last wave out zeroes the counters for the next launch.  Every
    // other wave has made its final claim and its final count before adding
    // itself to exit_count.
    uint32_t prev = 0;
    if (lane == 0) prev = __hip_atomic_fetch_add(exit_count, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
    prev = __builtin_amdgcn_readfirstlane(prev);
    const uint32_t total_waves = gridDim.x * kWavesPerBlock;
    if (prev == total_waves - 1) {
        for (int i = lane; i < count; i += kWave) __hip_atomic_store(&done[i], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (lane == 0) {
            __hip_atomic_store(ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(exit_count, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

}  // namespace

hipError_t launch_decode_m1(const DecodeEntry* table, int count, int total_tiles, int max_gpl, uint32_t* sync,
                            uint32_t spin_limit, int blocks, hipStream_t stream) {
    if (max_gpl <= 4) {
        hipLaunchKernelGGL((decode_m1_kernel<4>), dim3(blocks), dim3(kBlock), 0, stream, table, count,
                           total_tiles, sync, spin_limit);
    } else {
        hipLaunchKernelGGL((decode_m1_kernel<8>), dim3(blocks), dim3(kBlock), 0, stream, table, count,
                           total_tiles, sync, spin_limit);
    }
    return hipGetLastError();
}

}  // namespace wq
