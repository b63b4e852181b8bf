// wq_decode_linears_noalloc: the decode step for callers that cannot
// allocate (code under HIP graph capture, tight serving loops, harnesses
// that forbid hipMalloc).  Same planning, kernels and results as
// wq_decode_linears; the only difference is where the plan lives:
//
//   * on the device, in `scratch`, a fixed file-scope array of
//     WQ_NOALLOC_SCRATCH_BYTES per device, held until the process ends.  Its
//     device address comes from hipGetSymbolAddress, once per device, on the
//     first call made with that device current;
//   * it gets there through plan_write_kernel launches queued on the call's
//     stream ahead of the GEMV launches, whose kernel arguments carry the
//     plan bytes.  Nothing is copied from host memory at run time, so a
//     captured call records its plan by value and its graph replays
//     correctly whatever other calls wrote to the array in between;
//   * on the host, the planning works in fixed static storage guarded by a
//     mutex.
//
// Every call on a device shares that device's array and leaves its own plan
// there; the plan is rewritten in full by each call, so nothing has to start
// at zero.  Calls (or graph replays) that overlap in time on one device, on
// different streams, race on the array.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "wq_device.h"
#include "wq_plan.h"

namespace wq {
namespace {

using plan::BatchPlan;
using plan::Group;
using plan::GroupPlan;
using plan::PlanBuf;
using plan::Span;

constexpr size_t kScratchBytes = (size_t)WQ_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxLinears = (int)WQ_NOALLOC_MAX_LINEARS;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Plan bytes carried by one plan_write_kernel launch: 224 16-byte vectors,
// which keeps its arguments (3600 bytes) under the 4 KiB of a launch.
constexpr int kChunkVecs = 224;
struct PlanChunk {
    dev::u32x4* dst;
    uint32_t vecs;
    uint32_t pad;
    dev::u32x4 data[kChunkVecs];
};
static_assert(sizeof(PlanChunk) <= 3600, "plan chunk arguments");

__global__ __launch_bounds__(256) void plan_write_kernel(const PlanChunk c) {
    const int t = threadIdx.x;
    if (t < (int)c.vecs) c.dst[t] = c.data[t];
}

struct DeviceState {
    bool ready = false;
    unsigned char* ptr = nullptr;  // device address of `scratch` on this device
    plan::DeviceShape shape;
};

// Host-side storage of the calls, guarded by g_mu.
std::mutex g_mu;
DeviceState g_dev[kMaxDevices];
Span g_weights[2 * kMaxLinears];
Span g_reads[kMaxLinears], g_writes[kMaxLinears];
Group g_groups[kMaxLinears];
GroupPlan g_gplans[kMaxLinears];
BatchPlan g_bplans[kMaxLinears];
alignas(16) unsigned char g_plan[kScratchBytes];

wq_status fail(wq_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
wq_status fail(wq_status st, const char* fmt, ...) {
    char msg[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(msg, sizeof(msg), fmt, ap);
    va_end(ap);
    return record_error(st, msg);
}

// Set up `device` (current): the scratch array's device address and the
// device's wave capacities.
wq_status device_state(const char* fn, int device, DeviceState*& out) {
    if (device < 0 || device >= kMaxDevices)
        return fail(WQ_ERR_UNSUPPORTED, "%s: device %d beyond the %d devices supported", fn, device, kMaxDevices);
    DeviceState& d = g_dev[device];
    if (!d.ready) {
        void* p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_error(fn, e);
        if (!p) return fail(WQ_ERR_HIP, "%s: no device address for the scratch array", fn);
        if ((e = plan::device_shape(device, d.shape)) != hipSuccess) return hip_error(fn, e);
        d.ptr = static_cast<unsigned char*>(p);
        d.ready = true;
    }
    out = &d;
    return WQ_OK;
}

// Queue the plan bytes [0, size) for the scratch array at `dst`.
hipError_t write_plan(unsigned char* dst, const unsigned char* bytes, size_t size, hipStream_t stream) {
    PlanChunk c;
    for (size_t off = 0; off < size; off += sizeof(c.data)) {
        const size_t n = std::min(sizeof(c.data), size - off);  // a multiple of 16
        c.dst = reinterpret_cast<dev::u32x4*>(dst + off);
        c.vecs = (uint32_t)(n / 16);
        c.pad = 0;
        std::memcpy(c.data, bytes + off, n);
        hipLaunchKernelGGL(plan_write_kernel, dim3(1), dim3(256), 0, stream, c);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace
}  // namespace wq

extern "C" wq_status wq_decode_linears_noalloc(const wq_linear* linears, int64_t count, int64_t M, int64_t group,
                                               void* stream) {
    using namespace wq;
    static const char* fn = "wq_decode_linears_noalloc";
    if (!linears) return fail(WQ_ERR_INVALID_ARG, "%s: null descriptor array", fn);
    if (count <= 0 || count > kMaxLinears)
        return fail(WQ_ERR_INVALID_ARG, "%s: count must be in [1, %d] (WQ_NOALLOC_MAX_LINEARS; count=%lld)", fn,
                    kMaxLinears, (long long)count);
    std::lock_guard<std::mutex> guard(g_mu);
    wq_status st = check_decode_list(fn, linears, count, M, group, g_weights);
    if (st != WQ_OK) return st;
    (void)hipGetLastError();
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (M > kMaxSmallBatchM) {
        // Prompt-sized batches: one launch per linear, no plan.
        for (int64_t i = 0; i < count; ++i) {
            const wq_linear& l = linears[i];
            if ((st = hip_error(fn, launch_gemv(l.packed_w, l.scales, l.x, l.y, l.N, l.K, M, s))) != WQ_OK) return st;
        }
        return WQ_OK;
    }
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return hip_error(fn, e);
    DeviceState* ds = nullptr;
    if ((st = device_state(fn, device, ds)) != WQ_OK) return st;

    int ngroups = 0;
    {
        plan::SpanList reads(g_reads, kMaxLinears), writes(g_writes, kMaxLinears);
        plan::split_groups(linears, (int)count, M, reads, writes, [&](const Group& g) { g_groups[ngroups++] = g; });
    }
    const bool matrix = use_matrix_cores(M);
    const int64_t target = ds->shape.mb_waves[M <= 2 ? 0 : M <= 4 ? 1 : 2];
    PlanBuf pb{g_plan, kScratchBytes, 0, false};
    for (int i = 0; i < ngroups; ++i) {
        if (!g_groups[i].grouped) continue;
        if (M == 1) g_gplans[i] = plan::plan_group(linears, g_groups[i], ds->shape.blocks4, ds->shape.blocks8, pb);
        else if (matrix) g_bplans[i] = plan::plan_batch_group(linears, g_groups[i], pb);
        else g_bplans[i] = plan::plan_vector_group(linears, g_groups[i], target, pb);
    }
    if (pb.overflow)
        return fail(WQ_ERR_INVALID_ARG, "%s: the plan of these %lld linears exceeds the %zu-byte scratch array "
                    "(WQ_NOALLOC_SCRATCH_BYTES)", fn, (long long)count, kScratchBytes);
    if (pb.size > 0 && (e = write_plan(ds->ptr, g_plan, pb.size, s)) != hipSuccess) return hip_error(fn, e);
    return hip_error(fn, plan::launch_groups(linears, g_groups, ngroups, g_gplans, g_bplans, ds->ptr, M, matrix, s));
}
