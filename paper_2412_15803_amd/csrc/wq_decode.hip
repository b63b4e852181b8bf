// Grouped batch-1 GEMV: all linears of one dependency level of a decode step
// in a single launch (the per-token work of the paper's decode loop, Sec. 1
// and Table 1; kernel fusion across operators, Sec. 2.3).
//
// The host splits a decode step's linears into groups in which no linear
// reads or overwrites another's data; groups run in stream order, so inside a
// launch every linear is independent.  Linears are further sorted into shape
// classes (same lanes per row and groups per lane), each class's rows are cut
// into steps, and every workgroup of the grid is given one class and a
// contiguous, equal share of that class's steps (classes get workgroups in
// proportion to their bytes).  A workgroup is one CU's worth of waves (three
// per SIMD, or two for the wide variant), and its waves share the
// workgroup's range dynamically: the range is cut into chunks of a few
// steps, wave w starts on chunk w and then takes the next untaken chunk from
// a counter in LDS.  Waves that share a SIMD do not run at the same speed
// (the oldest one wins the issue arbitration: with equal static shares the
// youngest of three finished 1.6x later than the oldest), so the dynamic
// share keeps every wave busy until the range is done.  Chunks are taken in
// order, so a wave's chunks lie close together and it rarely changes linear.
//
// Inside a chunk a wave streams its steps through a loop specialised for its
// class's shape: two to four register buffers (compute a buffer, refill it
// with the step that many ahead, go on to the next), so later steps' weights
// -- of this chunk or the next one -- are always in flight while the current
// step is computed.  Outputs are staged in LDS and written once per run of
// contiguous rows.  No global atomics, no waiting between workgroups.
#include "wq_device.h"
#include "wq_internal.h"

namespace wq {
namespace {

using namespace dev;

// Waves of one workgroup (one workgroup per CU): two per SIMD for the
// narrow (MAXG <= 4) and the wide variant.  The narrow variant took three
// per SIMD with three buffers of six-load steps; two per SIMD with two
// buffers of four-load steps measured faster on the 3B step (272-274 against
// 281-282 us over 200 steps, alternated on one box) and on one-layer calls
// (3B 14.4-15.3 against 17.2 us).
#ifndef WQ_GROUPED_WAVES4
#define WQ_GROUPED_WAVES4 8
#endif
#ifndef WQ_GROUPED_WAVES8
#define WQ_GROUPED_WAVES8 8
#endif
__host__ __device__ constexpr int cu_waves(int maxg) { return maxg <= 4 ? WQ_GROUPED_WAVES4 : WQ_GROUPED_WAVES8; }

// What computing a step needs (the linear, its rows, its groups per row);
// issuing it also needs the linear's pointers, which the step iterator holds
// for the linear it is in.  Steps, rows and step counts are 32-bit: a
// launch's classes have fewer than 2^31 steps (the host splits larger groups)
// and a linear read through buffer offsets fewer than 2^28 rows.
struct Step {
    int lin;    // -1 once the wave's work is done
    int nrows;  // rows of this step inside its linear
    int row;    // first row
    int ng;
};

// The current linear of a wave's walk.
struct LinearRef {
    int lin;
    int ng;
    int n;                   // rows, for the last step's row count
    uint32_t scale_bytes;    // n * ng * 2: extent of the scales (codes: 8x)
    const void* packed;
    const uint16_t* scales;
};

// Walks a wave's chunks of one workgroup's share of a class: steps are
// numbered per class in linear order, each linear owning steps [first_step,
// first_step + steps); the chunks of one share are taken in increasing
// order, so within a share the walk only moves forward through the class's
// list.  The current linear's fields are cached and reloaded only at a
// boundary.
struct StepIter {
    int idx;          // position in the class's linear list
    int pos;          // next step (class numbering)
    int end;          // one past the last step of the current chunk
    int first_step;   // of the current linear
    int lin_end;      // first step of the next linear
    int begin, end_all;  // the workgroup's share of the class
    int cs;              // its steps per chunk
    bool done;
    uint32_t next_chunk;  // the chunk this wave takes next
    LinearRef cur;
};

// The next untaken chunk of the workgroup (one LDS atomic, wave-uniform).
__device__ __forceinline__ uint32_t take_chunk(uint32_t* counter, int lane) {
    uint32_t v = 0;
    if (lane == 0) v = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    return __builtin_amdgcn_readfirstlane(v);
}

__device__ __forceinline__ void load_linear(StepIter& it, const DecodePlan& p, const DecodeClass& c) {
    const int lin = p.class_lin[c.first + it.idx];
    const DecodeEntry& e = p.entries[lin];
    it.cur.lin = lin;
    it.cur.ng = e.ng;
    it.cur.n = (int)e.n;
    it.cur.packed = e.packed;
    it.cur.scales = e.scales;
    it.cur.scale_bytes = (uint32_t)(e.n * e.ng * 2);
    it.first_step = (int)e.first_step;
    it.lin_end = (int)(e.first_step + e.steps);
}

// Move to the wave's next chunk of the workgroup's share.  Returns false
// once the share is done.
__device__ __forceinline__ bool next_chunk(StepIter& it, uint32_t* lds_counter, int lane) {
    const int64_t start = it.begin + (int64_t)it.next_chunk * it.cs;
    if (start >= it.end_all) return false;
    it.pos = (int)start;
    it.end = min(it.pos + it.cs, it.end_all);
    it.next_chunk = take_chunk(lds_counter, lane);
    return true;
}

template <int R>
__device__ __forceinline__ Step next_step(StepIter& it, const DecodePlan& p, const DecodeClass& c,
                                          uint32_t* lds_counter, int lane) {
    Step s;
    if (it.pos >= it.end && (it.done || !next_chunk(it, lds_counter, lane))) {
        it.done = true;  // stay done without taking more chunks
        it.pos = it.end;
        s.lin = -1;
        s.nrows = 0;
        s.row = 0;
        s.ng = it.cur.ng;
        return s;
    }
    // Chunks only move forward, so the walk to the chunk's linear does too.
    while (it.pos >= it.lin_end) {
        ++it.idx;
        load_linear(it, p, c);
    }
    s.lin = it.cur.lin;
    s.ng = it.cur.ng;
    s.row = (it.pos - it.first_step) * R;
    s.nrows = min(R, it.cur.n - s.row);
    ++it.pos;
    return s;
}

// The wave's x registers, the linear they belong to, and a run of
// contiguous rows of that linear's y staged in LDS ([ybase, yend) of y).
// The staged rows are written out when the next step's rows do not continue
// them (a new chunk elsewhere, another linear) or would overflow the slice.
// x is switched when the wave computes the first step of another linear: the
// fresh x loads are the youngest in flight, so the wave waits for its
// pipeline once per linear it enters.
template <int MAXG>
struct XSlot {
    half2v xr[MAXG][16];
    int lin;
    uint16_t* y;
    int ybase, yend;
};

// Write the `count` staged rows ylds[0, count) to y[row0, row0 + count)
// through a buffer resource (one offset register per lane: this runs while
// the pipeline's buffers and x are live).
__device__ __forceinline__ void flush_run(uint16_t* y, int row0, const uint16_t* ylds, int count, int lane) {
    wave_lds_sync();
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc(y + row0, (short)0, count * 2, kRawBufferFlags);
    for (int i = lane; i < count; i += kWave)
        __builtin_amdgcn_raw_buffer_store_b16(ylds[i], r, (uint32_t)i * 2u, 0, 0);
    wave_lds_sync();  // stores have read the slice before it is refilled
}

// x and y of the linear a step belongs to are read from the plan only when
// the wave enters that linear.
template <int LPR, int GPL, int MAXG>
__device__ __forceinline__ void compute_from(const StepBuf& b, XSlot<MAXG>& xs, const Step& s,
                                             const DecodePlan& p, uint16_t* ylds, int lane) {
    if (s.lin < 0) return;
    const bool new_lin = xs.lin != s.lin;
    if (new_lin || s.row != xs.yend || s.row + s.nrows - xs.ybase > kYRows) {
        if (xs.lin >= 0) flush_run(xs.y, xs.ybase, ylds, xs.yend - xs.ybase, lane);
        if (new_lin) {
            const DecodeEntry& e = p.entries[s.lin];
            load_x_lane<LPR, GPL, MAXG>(e.x, s.ng, lane, xs.xr);
            xs.lin = s.lin;
            xs.y = e.y;
        }
        xs.ybase = s.row;
    }
    compute_step<LPR, GPL, MAXG, grouped_step_loads(MAXG)>(b, xs.xr, s.nrows, ylds, s.row - xs.ybase, lane);
    xs.yend = s.row + s.nrows;
}

// Issues are unconditional: once the wave's work is done it re-loads row 0
// of its current linear (never computed), so every path through the loop
// issues the same loads and the compiler's wait counts stay exact.
template <int LPR, int GPL, int MAXG>
__device__ __forceinline__ void issue_from(StepBuf& b, const Step& s, const LinearRef& l, int lane) {
    issue_step<LPR, GPL, kCpolNonTemporal, grouped_step_loads(MAXG)>(b, make_rsrc(l.packed, l.scales, l.scale_bytes),
                                                                     s.row, l.ng, lane);
}

// Register buffers in the pipeline: as many steps as fit a budget of
// in-flight 16-byte loads per lane (8 in the narrow kernel, which gives the
// 3B step's K = 3072 and 8192 linears two buffers; 14 beside the wide one's
// x registers), at least two and at most four.
#ifndef WQ_DEPTH_BUDGET4
#define WQ_DEPTH_BUDGET4 8
#endif
#ifndef WQ_DEPTH_BUDGET8
#define WQ_DEPTH_BUDGET8 14
#endif
template <int LPR, int GPL, int MAXG>
constexpr int pipeline_depth() {
    constexpr int per_step = StepShape<LPR, GPL, grouped_step_loads(MAXG)>::U * GPL;
    constexpr int nb = (MAXG <= 4 ? WQ_DEPTH_BUDGET4 : WQ_DEPTH_BUDGET8) / per_step;
    return nb < 2 ? 2 : (nb > 4 ? 4 : nb);
}

// Steps per chunk: up to twice the pipeline depth (a wave's loads of the
// next chunk are then issued while half of the current one is still to be
// computed), fewer when the workgroup's range would give its waves fewer
// than WQ_CHUNKS_PER_WAVE chunks each.  Short launches (one layer per call)
// thus hand out smaller chunks and end more evenly: the 3B layer call took
// 13.7-13.8 us with three chunks per wave against 14.6-14.9 us with one (the
// full step, whose chunks stay at the maximum, is unchanged).
#ifndef WQ_CHUNKS_PER_WAVE
#define WQ_CHUNKS_PER_WAVE 3
#endif
template <int LPR, int GPL, int MAXG>
__device__ __forceinline__ int chunk_steps(int range, int waves) {
    constexpr int kMax = 2 * pipeline_depth<LPR, GPL, MAXG>();
    return max(1, min(kMax, range / (waves * WQ_CHUNKS_PER_WAVE)));
}

// One wave's share of its workgroup's steps: chunk `wave` first, then
// whatever chunk the counter hands out next.
template <int LPR, int GPL, int MAXG>
__device__ __forceinline__ void run_block(const DecodePlan& p, const DecodeClass& c, const DecodeBlock& b,
                                          uint32_t* lds_counter, int wave, int waves, uint16_t* ylds, int lane) {
    constexpr int NB = pipeline_depth<LPR, GPL, MAXG>();
    constexpr int R = StepShape<LPR, GPL, grouped_step_loads(MAXG)>::ROWS;
    static_assert(2 * NB * R <= kYRows, "a chunk's rows fit the wave's staging slice");
    StepIter it;
    it.begin = b.begin;
    it.end_all = b.end;
    it.cs = chunk_steps<LPR, GPL, MAXG>(b.end - b.begin, waves);
    it.done = false;
    it.next_chunk = (uint32_t)wave;
    if (!next_chunk(it, lds_counter, lane)) return;  // fewer chunks than waves
    // The linear holding the workgroup's first step comes with the plan; the
    // wave's first chunk is at most a few steps further.
    it.idx = b.pos;
    load_linear(it, p, c);
    // x of the linear holding the wave's first step is loaded before any
    // weight load.  Loaded later (when that step is computed, as for the
    // linears the wave enters afterwards), it would be the youngest load in
    // flight and the first computation would wait for the whole pipeline:
    // in a one-layer call that is most of a wave's work, and its compute
    // then followed all of its data instead of overlapping it.
    while (it.pos >= it.lin_end) {
        ++it.idx;
        load_linear(it, p, c);
    }
    XSlot<MAXG> xs;
    u32x4 xraw[MAXG][4];
    const int xng = it.cur.ng;
    {
        const DecodeEntry& e = p.entries[it.cur.lin];
        load_x_raw<LPR, GPL, MAXG>(e.x, xng, lane, xraw);
        load_order_fence();
        xs.lin = it.cur.lin;
        xs.y = e.y;
        xs.ybase = xs.yend = (it.pos - it.first_step) * R;
    }
    // The first pass only issues (x's round trip overlaps these loads, and
    // x is paired after them); afterwards each pass computes the step a
    // buffer holds and refills that buffer with the wave's next step.
    StepBuf buf[NB];
    Step st[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
        st[i] = next_step<R>(it, p, c, lds_counter, lane);
        issue_from<LPR, GPL, MAXG>(buf[i], st[i], it.cur, lane);
    }
    pair_x<LPR, GPL, MAXG>(xraw, xng, lane, xs.xr);
    for (;;) {
        bool any = false;
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            compute_from<LPR, GPL, MAXG>(buf[i], xs, st[i], p, ylds, lane);
            st[i] = next_step<R>(it, p, c, lds_counter, lane);
            any = any || st[i].lin >= 0;
            issue_from<LPR, GPL, MAXG>(buf[i], st[i], it.cur, lane);
        }
        if (!any) break;
    }
    if (xs.lin >= 0) flush_run(xs.y, xs.ybase, ylds, xs.yend - xs.ybase, lane);
}

// The (lanes per row, groups per lane) shapes a launch supports: those with
// at most MAXG groups per lane.
#define WQ_SHAPES_4(X) X(64, 1) X(64, 2) X(64, 3) X(64, 4) X(32, 1) X(32, 3) X(16, 1) X(16, 3)
#define WQ_SHAPES_8(X) WQ_SHAPES_4(X) X(64, 5) X(64, 6) X(64, 7) X(64, 8) X(32, 5) X(32, 7) X(16, 5) X(16, 7)

// The plan arrays arrive as separate read-only, non-aliasing arguments, so
// every table read is a scalar load with a wave-uniform value.  One
// workgroup per CU, two waves per SIMD (cu_waves).
template <int MAXG>
__global__ __launch_bounds__(cu_waves(MAXG) * kWave, cu_waves(MAXG) / 4) void grouped_m1_kernel(
    const DecodeEntry* __restrict__ entries, const DecodeClass* __restrict__ classes,
    const int32_t* __restrict__ class_lin, const DecodeBlock* __restrict__ blocks, int nclasses) {
    constexpr int kWaves = cu_waves(MAXG);
    __shared__ __align__(16) uint16_t s_y[kWaves][kYRows];
    __shared__ uint32_t s_chunk;
    if (threadIdx.x == 0) s_chunk = kWaves;  // chunks 0 .. kWaves - 1 are the waves' first
    __syncthreads();
    DecodePlan p;
    p.entries = entries;
    p.classes = classes;
    p.class_lin = class_lin;
    p.blocks = blocks;
    p.nclasses = nclasses;
    const int lane = threadIdx.x & (kWave - 1);
    // The wave index is the same in every lane; saying so keeps everything
    // derived from it in scalar registers and all branches uniform.
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int blk = blockIdx.x;
    int ci = -1;
    for (int k = 0; k < nclasses; ++k)
        if (classes[k].blocks_begin <= blk && blk < classes[k].blocks_begin + classes[k].blocks) ci = k;
    if (ci < 0) return;
    const DecodeClass& c = classes[ci];
    const DecodeBlock& b = blocks[blk];
    if (b.begin >= b.end) return;
    uint16_t* ylds = s_y[wave];
#define WQ_RUN(L, G) \
    if (c.lpr == L && c.gpl == G) { run_block<L, G, MAXG>(p, c, b, &s_chunk, wave, kWaves, ylds, lane); return; }
    if constexpr (MAXG <= 4) {
        WQ_SHAPES_4(WQ_RUN)
    } else {
        WQ_SHAPES_8(WQ_RUN)
    }
#undef WQ_RUN
}

}  // namespace

hipError_t launch_grouped_m1(const DecodePlan& plan, int max_gpl, int blocks, hipStream_t stream) {
    if (max_gpl <= 4) {
        hipLaunchKernelGGL((grouped_m1_kernel<4>), dim3(blocks), dim3(cu_waves(4) * kWave), 0, stream,
                           plan.entries, plan.classes, plan.class_lin, plan.blocks, plan.nclasses);
    } else {
        hipLaunchKernelGGL((grouped_m1_kernel<8>), dim3(blocks), dim3(cu_waves(8) * kWave), 0, stream,
                           plan.entries, plan.classes, plan.class_lin, plan.blocks, plan.nclasses);
    }
    return hipGetLastError();
}

hipError_t grouped_capacity(int max_gpl, int device, int& blocks) {
    int per_cu = 0, cus = 0;
    hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess) return e;
    if (max_gpl <= 4)
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, grouped_m1_kernel<4>, cu_waves(4) * kWave, 0);
    else
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, grouped_m1_kernel<8>, cu_waves(8) * kWave, 0);
    if (e != hipSuccess) return e;
    blocks = (per_cu > 0 ? per_cu : 1) * (cus > 0 ? cus : 1);
    return hipSuccess;
}

}  // namespace wq
