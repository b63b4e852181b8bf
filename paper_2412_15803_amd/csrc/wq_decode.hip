// Grouped batch-1 GEMV: all linears of one dependency level of a decode step
// in a single launch (the per-token work of the paper's decode loop, Sec. 1
// and Table 1; kernel fusion across operators, Sec. 2.3).
//
// The host splits a decode step's linears into groups in which no linear
// reads or overwrites another's data; groups run in stream order, so inside a
// launch every linear is independent.  Linears are further sorted into shape
// classes (same lanes per row and groups per lane), each class's rows are cut
// into steps, and every wave of the grid is given one class and a contiguous,
// equal share of that class's steps (classes get waves in proportion to
// their bytes).  A wave therefore streams one long contiguous range of rows,
// crossing linear boundaries only where its range does, through a loop
// specialised for its class's shape: two or three register buffers (compute
// a buffer, refill it with the step that many ahead, go on to the next), so
// later steps' weights -- of this linear or the next one -- are always in
// flight while the current step is computed.  Outputs are staged in LDS and
// written per linear.  No atomics, no waiting between waves.
#include "wq_device.h"
#include "wq_internal.h"

namespace wq {
namespace {

using namespace dev;

constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / kWave;

// One step as the pipeline sees it: everything needed to issue and compute
// it, so the steady state reads no table entries.
struct Step {
    int lin;                 // -1 past the end of the wave's range
    int nrows;               // rows of this step inside its linear
    int ng;
    uint32_t scale_bytes;    // n * ng * 2: extent of the scales (codes: 8x)
    int64_t row;             // first row
    const void* packed;
    const uint16_t* scales;
};

// Walks the wave's step range [pos, end) of a class: steps are numbered per
// class in linear order, each linear owning steps [first_step, first_step +
// steps), so the walk only ever moves forward through the class's list.  The
// current linear's fields are cached and reloaded only at a boundary.
struct StepIter {
    int idx;        // position in the class's linear list
    int64_t pos;    // next step (class numbering)
    int64_t end;    // one past the wave's last step
    int64_t lin_end;  // first step of the next linear
    Step cur;       // fields of the current linear (row = its first step's row base)
    int64_t first_step;
};

__device__ __forceinline__ void load_linear(StepIter& it, const DecodePlan& p, const DecodeClass& c) {
    const int lin = p.class_lin[c.first + it.idx];
    const DecodeEntry& e = p.entries[lin];
    it.cur.lin = lin;
    it.cur.ng = e.ng;
    it.cur.row = e.n;  // rows of the linear, for the last step's row count
    it.cur.packed = e.packed;
    it.cur.scales = e.scales;
    it.cur.scale_bytes = (uint32_t)(e.n * e.ng * 2);
    it.first_step = e.first_step;
    it.lin_end = e.first_step + e.steps;
}

template <int R>
__device__ __forceinline__ Step next_step(StepIter& it, const DecodePlan& p, const DecodeClass& c) {
    Step s = it.cur;
    if (it.pos >= it.end) {
        s.lin = -1;
        return s;
    }
    while (it.pos >= it.lin_end) {
        ++it.idx;
        load_linear(it, p, c);
        s = it.cur;
    }
    const int64_t n = it.cur.row;
    s.row = (it.pos - it.first_step) * R;
    s.nrows = (int)min((int64_t)R, n - s.row);
    ++it.pos;
    return s;
}

// The wave's x registers, the linear they belong to, and the rows of that
// linear's y staged in LDS ([ybase, yend) of y).  x is switched when the wave
// computes the first step of another linear: the staged rows of the previous
// one are written out, and the fresh x loads are the youngest in flight, so
// the wave waits for its pipeline once per linear it enters.
template <int MAXG>
struct XSlot {
    half2v xr[MAXG][16];
    int lin;
    uint16_t* y;
    int64_t ybase, yend;
};

// x and y of the linear a step belongs to are read from the plan only when
// the wave enters that linear.
template <int LPR, int GPL, int MAXG>
__device__ __forceinline__ void compute_from(const StepBuf& b, XSlot<MAXG>& xs, const Step& s,
                                             const DecodePlan& p, uint16_t* ylds, int lane) {
    if (s.lin < 0) return;
    if (xs.lin != s.lin) {
        if (xs.lin >= 0) flush_y(xs.y, xs.ybase, ylds, (int)(xs.yend - xs.ybase), lane);
        const DecodeEntry& e = p.entries[s.lin];
        load_x_lane<LPR, GPL, MAXG>(e.x, s.ng, lane, xs.xr);
        xs.lin = s.lin;
        xs.y = e.y;
        xs.ybase = s.row;
    }
    compute_step<LPR, GPL, MAXG>(b, xs.xr, s.nrows, ylds, (int)(s.row - xs.ybase), lane);
    xs.yend = s.row + s.nrows;
}

// Issues are unconditional: past the end of the range the wave re-loads its
// last valid step (never computed), so every path through the loop issues
// the same loads and the compiler's wait counts stay exact.
template <int LPR, int GPL>
__device__ __forceinline__ void issue_from(StepBuf& b, const Step& s, int lane) {
    issue_step<LPR, GPL, kCpolNonTemporal>(b, make_rsrc(s.packed, s.scales, s.scale_bytes), s.row, s.ng, lane);
}

// Register buffers in the pipeline: as many steps as fit a budget of
// in-flight 16-byte loads per lane (18 beside the narrow kernel's x
// registers, which keeps three waves per SIMD; 14 beside the wide one's),
// at least two and at most four.
#ifndef WQ_DEPTH_BUDGET4
#define WQ_DEPTH_BUDGET4 18
#endif
#ifndef WQ_DEPTH_BUDGET8
#define WQ_DEPTH_BUDGET8 14
#endif
template <int LPR, int GPL, int MAXG>
constexpr int pipeline_depth() {
    constexpr int per_step = StepShape<LPR, GPL>::U * GPL;
    constexpr int nb = (MAXG <= 4 ? WQ_DEPTH_BUDGET4 : WQ_DEPTH_BUDGET8) / per_step;
    return nb < 2 ? 2 : (nb > 4 ? 4 : nb);
}

// The plan keeps every wave's range at most kYRows / R steps, so the staged
// rows of one linear always fit the wave's LDS slice.
template <int LPR, int GPL, int MAXG>
__device__ __forceinline__ void run_range(const DecodePlan& p, const DecodeClass& c, int64_t begin, int64_t end,
                                          uint16_t* ylds, int lane) {
    constexpr int R = StepShape<LPR, GPL>::ROWS;
    constexpr int NB = pipeline_depth<LPR, GPL, MAXG>();
    StepIter it;
    it.pos = begin;
    it.end = end;
    // Find the linear holding step `begin` (the class lists are short, a
    // forward scan is enough).
    it.idx = 0;
    load_linear(it, p, c);
    while (begin >= it.lin_end) {
        ++it.idx;
        load_linear(it, p, c);
    }
    XSlot<MAXG> xs;
    xs.lin = -1;
    xs.y = nullptr;
    xs.ybase = xs.yend = 0;
    StepBuf buf[NB];
    Step st[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) st[i].lin = -1;
    // The first pass only issues; afterwards each pass computes the step a
    // buffer holds and refills that buffer with the wave's next step.
    Step last = it.cur;  // the latest valid step (the range is never empty)
    for (;;) {
        bool any = false;
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            compute_from<LPR, GPL, MAXG>(buf[i], xs, st[i], p, ylds, lane);
            st[i] = next_step<R>(it, p, c);
            if (st[i].lin >= 0) last = st[i];
            any = any || st[i].lin >= 0;
            issue_from<LPR, GPL>(buf[i], st[i].lin >= 0 ? st[i] : last, lane);
        }
        if (!any) break;
    }
    if (xs.lin >= 0) flush_y(xs.y, xs.ybase, ylds, (int)(xs.yend - xs.ybase), lane);
}

// The (lanes per row, groups per lane) shapes a launch supports: those with
// at most MAXG groups per lane.
#define WQ_SHAPES_4(X) X(64, 1) X(64, 2) X(64, 3) X(64, 4) X(32, 1) X(32, 3) X(16, 1) X(16, 3)
#define WQ_SHAPES_8(X) WQ_SHAPES_4(X) X(64, 5) X(64, 6) X(64, 7) X(64, 8) X(32, 5) X(32, 7) X(16, 5) X(16, 7)

// The plan arrays arrive as separate read-only, non-aliasing arguments, so
// every table read is a scalar load with a wave-uniform value.
// Three waves per SIMD fit the narrow variant without spilling; the wide
// one (up to eight groups of x per lane) stays at two.
template <int MAXG>
__global__ __launch_bounds__(kBlock, MAXG <= 4 ? 3 : 2) void grouped_m1_kernel(const DecodeEntry* __restrict__ entries,
                                                            const DecodeClass* __restrict__ classes,
                                                            const int32_t* __restrict__ class_lin, int nclasses) {
    DecodePlan p;
    p.entries = entries;
    p.classes = classes;
    p.class_lin = class_lin;
    p.nclasses = nclasses;
    const int lane = threadIdx.x & (kWave - 1);
    // The wave index is the same in every lane; saying so keeps everything
    // derived from it in scalar registers and all branches uniform.
    const int wave = __builtin_amdgcn_readfirstlane(blockIdx.x * kWavesPerBlock + threadIdx.x / kWave);
    int ci = -1;
    for (int k = 0; k < nclasses; ++k)
        if (classes[k].waves_begin <= wave && wave < classes[k].waves_begin + classes[k].waves) ci = k;
    if (ci < 0) return;
    const DecodeClass& c = classes[ci];
    const int64_t i = wave - c.waves_begin;
    const int64_t begin = i * c.steps / c.waves;
    const int64_t end = (i + 1) * c.steps / c.waves;
    if (begin >= end) return;
    __shared__ __align__(16) uint16_t s_y[kWavesPerBlock][kYRows];
    uint16_t* ylds = s_y[threadIdx.x / kWave];
#define WQ_RUN(L, G) \
    if (c.lpr == L && c.gpl == G) { run_range<L, G, MAXG>(p, c, begin, end, ylds, lane); return; }
    if constexpr (MAXG <= 4) {
        WQ_SHAPES_4(WQ_RUN)
    } else {
        WQ_SHAPES_8(WQ_RUN)
    }
#undef WQ_RUN
}

}  // namespace

hipError_t launch_grouped_m1(const DecodePlan& plan, int max_gpl, int waves, hipStream_t stream) {
    const int blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
    if (max_gpl <= 4) {
        hipLaunchKernelGGL((grouped_m1_kernel<4>), dim3(blocks), dim3(kBlock), 0, stream, plan.entries,
                           plan.classes, plan.class_lin, plan.nclasses);
    } else {
        hipLaunchKernelGGL((grouped_m1_kernel<8>), dim3(blocks), dim3(kBlock), 0, stream, plan.entries,
                           plan.classes, plan.class_lin, plan.nclasses);
    }
    return hipGetLastError();
}

hipError_t grouped_capacity(int max_gpl, int device, int& waves) {
    int per_cu = 0, cus = 0;
    hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
    if (e != hipSuccess) return e;
    if (max_gpl <= 4)
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, grouped_m1_kernel<4>, kBlock, 0);
    else
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, grouped_m1_kernel<8>, kBlock, 0);
    if (e != hipSuccess) return e;
    waves = (per_cu > 0 ? per_cu : 1) * (cus > 0 ? cus : 1) * kWavesPerBlock;
    return hipSuccess;
}

}  // namespace wq
