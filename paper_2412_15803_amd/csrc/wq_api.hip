// C ABI of the 4-bit decode-linear library: argument validation (entirely on
// the host, before any HIP call), kernel dispatch, and error reporting.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <utility>
#include <vector>

#include "wq.h"
#include "wq_device.h"
#include "wq_internal.h"
#include "wq_plan.h"

namespace {

thread_local char g_last_error[512] = "no error";

wq_status fail(wq_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return st;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

using wq::plan::overlaps;
using wq::plan::Span;
using wq::plan::span_of;

// N, K, group checks shared by every entry point.
wq_status check_shape(const char* fn, int64_t n, int64_t k, int64_t group) {
    if (n <= 0 || k <= 0) return fail(WQ_ERR_INVALID_ARG, "%s: N and K must be positive (N=%lld K=%lld)", fn, (long long)n, (long long)k);
    if (group != 32) return fail(WQ_ERR_UNSUPPORTED, "%s: only group=32 is supported (got %lld)", fn, (long long)group);
    if (k % 32 != 0) return fail(WQ_ERR_UNSUPPORTED, "%s: K must be a multiple of 32 (K=%lld)", fn, (long long)k);
    if (n > WQ_MAX_N || k > WQ_MAX_K) return fail(WQ_ERR_INVALID_ARG, "%s: N or K too large (N=%lld K=%lld)", fn, (long long)n, (long long)k);
    // Keep every byte count below 2^62.
    if (n > (((int64_t)1 << 62) / 4) / k) return fail(WQ_ERR_INVALID_ARG, "%s: N*K too large", fn);
    return WQ_OK;
}

struct GemvArgs {
    const uint32_t* packed;
    const uint16_t* scales;
    const uint16_t* x;
    uint16_t* y;
    int64_t n, k;
};

wq_status check_gemv(const char* fn, const GemvArgs& a, int64_t m, int64_t group) {
    if (!a.packed || !a.scales || !a.x || !a.y) return fail(WQ_ERR_INVALID_ARG, "%s: null pointer", fn);
    if (m <= 0 || m > WQ_MAX_M) return fail(WQ_ERR_INVALID_ARG, "%s: M must be in [1, %lld] (M=%lld)", fn, (long long)WQ_MAX_M, (long long)m);
    const wq_status st = check_shape(fn, a.n, a.k, group);
    if (st != WQ_OK) return st;
    if (!aligned(a.packed, 16)) return fail(WQ_ERR_MISALIGNED, "%s: packed_w must be 16-byte aligned", fn);
    if (!aligned(a.x, 16)) return fail(WQ_ERR_MISALIGNED, "%s: x must be 16-byte aligned", fn);
    if (!aligned(a.scales, 2)) return fail(WQ_ERR_MISALIGNED, "%s: scales must be 2-byte aligned", fn);
    if (!aligned(a.y, 2)) return fail(WQ_ERR_MISALIGNED, "%s: y must be 2-byte aligned", fn);
    const Span y = span_of(a.y, 2 * m * a.n);
    if (overlaps(y, span_of(a.x, 2 * m * a.k)) || overlaps(y, span_of(a.packed, a.n * a.k / 2)) ||
        overlaps(y, span_of(a.scales, a.n * (a.k / 32) * 2)))
        return fail(WQ_ERR_INVALID_ARG, "%s: y overlaps x, packed_w or scales", fn);
    return WQ_OK;
}

wq_status hip_status(const char* fn, hipError_t e) {
    if (e == hipSuccess) return WQ_OK;
    return fail(WQ_ERR_HIP, "%s: HIP error %d (%s)", fn, (int)e, hipGetErrorString(e));
}


// ------------------------------------------------------------ decode step

using wq::plan::BatchPlan;
using wq::plan::Group;
using wq::plan::GroupPlan;
using wq::plan::PlanBuf;

// Library-owned resources of wq_decode_linears, per (device, stream) pair
// the function is called with, kept until the process ends:
//   * device plan buffers, one per recently used descriptor list: up to
//     kPlanSlots that later calls may reuse, plus any number that a stream
//     capture recorded launches against, which are frozen (never rewritten or
//     freed, so the captured graph stays valid);
//   * two pinned host staging buffers, each with an event recorded after the
//     upload it holds, so that uploading a new list blocks the host only when
//     both still hold uploads the device has not read;
//   * the device's resident-wave capacities.
constexpr int kPlanSlots = 32;

struct PlanSlot {
    unsigned char* d = nullptr;
    size_t cap = 0;
    std::vector<unsigned char> bytes;  // the plan the buffer holds
    size_t extra = 0;                  // zeroed device bytes after it (device-owned state)
    bool frozen = false;
    uint64_t last_use = 0;
};

struct Stage {
    unsigned char* h = nullptr;
    size_t cap = 0;
    hipEvent_t read = nullptr;  // recorded on the stream after the copy from h
    bool pending = false;
    uint64_t seq = 0;
};

struct DecodeWorkspace {
    std::vector<PlanSlot> slots;
    Stage stage[2];
    wq::plan::DeviceShape shape;
    uint64_t clock = 0;
};

std::mutex g_ws_mu;
std::map<std::pair<int, hipStream_t>, DecodeWorkspace*> g_ws;

wq_status get_workspace(const char* fn, hipStream_t stream, DecodeWorkspace*& out) {
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return hip_status(fn, e);
    DecodeWorkspace*& ws = g_ws[std::make_pair(device, stream)];
    if (!ws) {
        std::unique_ptr<DecodeWorkspace> fresh(new DecodeWorkspace());
        for (Stage& st : fresh->stage)
            if ((e = hipEventCreateWithFlags(&st.read, hipEventDisableTiming)) != hipSuccess) return hip_status(fn, e);
        if ((e = wq::plan::device_shape(device, fresh->shape)) != hipSuccess) return hip_status(fn, e);
        ws = fresh.release();
    }
    out = ws;
    return WQ_OK;
}

size_t align16(size_t v) { return (v + 15) & ~size_t(15); }

size_t pow2_at_least(size_t v) {
    size_t cap = 4096;
    while (cap < v) cap *= 2;
    return cap;
}

// A staging buffer of at least `bytes` that the device no longer reads.
wq_status take_stage(const char* fn, DecodeWorkspace* ws, size_t bytes, Stage*& out) {
    hipError_t e;
    for (Stage& st : ws->stage) {
        if (st.pending) {
            e = hipEventQuery(st.read);
            if (e == hipSuccess) st.pending = false;
            else if (e != hipErrorNotReady) return hip_status(fn, e);
        }
    }
    Stage* st = nullptr;
    for (Stage& c : ws->stage)
        if (!c.pending && (!st || c.cap > st->cap)) st = &c;
    if (!st) {
        // Both still hold uploads in flight: wait for the older one.
        st = ws->stage[0].seq <= ws->stage[1].seq ? &ws->stage[0] : &ws->stage[1];
        if ((e = hipEventSynchronize(st->read)) != hipSuccess) return hip_status(fn, e);
        st->pending = false;
    }
    if (st->cap < bytes) {
        if (st->h) (void)hipHostFree(st->h);
        st->h = nullptr;
        st->cap = 0;
        const size_t cap = pow2_at_least(bytes);
        if ((e = hipHostMalloc(reinterpret_cast<void**>(&st->h), cap)) != hipSuccess) return hip_status(fn, e);
        st->cap = cap;
    }
    out = st;
    return WQ_OK;
}

// The device address of a buffer holding `bytes`: a resident copy of the
// same plan if there is one, else a fresh upload into a free or the least
// recently used reusable slot (stream-ordered, so launches already queued
// on this stream read the old contents).  Under stream capture only a
// resident plan is accepted, and its slot is frozen.
wq_status place_plan(const char* fn, DecodeWorkspace* ws, const std::vector<unsigned char>& bytes,
                     hipStream_t stream, bool capturing, const unsigned char*& d_plan, size_t extra = 0) {
    const uint64_t now = ++ws->clock;
    for (PlanSlot& s : ws->slots) {
        if (s.extra == extra && s.bytes == bytes) {
            s.last_use = now;
            if (capturing) s.frozen = true;
            d_plan = s.d;
            return WQ_OK;
        }
    }
    if (capturing)
        return fail(WQ_ERR_UNSUPPORTED,
                    "%s: the stream is capturing and this descriptor list's plan is not on the device; make the "
                    "same call once on this stream outside capture first, or use wq_decode_linears_noalloc", fn);
    int reusable = 0;
    PlanSlot* slot = nullptr;
    for (PlanSlot& s : ws->slots) {
        if (s.frozen) continue;
        ++reusable;
        if (!slot || s.last_use < slot->last_use) slot = &s;
    }
    if (reusable < kPlanSlots) {
        ws->slots.emplace_back();
        slot = &ws->slots.back();
    }
    hipError_t e;
    const size_t need = align16(bytes.size()) + extra;
    if (slot->cap < need) {
        if (slot->d) {
            // Launches queued on this stream may still read the old buffer.
            if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_status(fn, e);
            (void)hipFree(slot->d);
        }
        slot->d = nullptr;
        slot->cap = 0;
        slot->bytes.clear();
        const size_t cap = pow2_at_least(need);
        if ((e = hipMalloc(reinterpret_cast<void**>(&slot->d), cap)) != hipSuccess) return hip_status(fn, e);
        slot->cap = cap;
    }
    Stage* st = nullptr;
    wq_status rs = take_stage(fn, ws, bytes.size(), st);
    if (rs != WQ_OK) return rs;
    std::memcpy(st->h, bytes.data(), bytes.size());
    if ((e = hipMemcpyAsync(slot->d, st->h, bytes.size(), hipMemcpyHostToDevice, stream)) != hipSuccess)
        return hip_status(fn, e);
    if ((e = hipEventRecord(st->read, stream)) != hipSuccess) return hip_status(fn, e);
    if (extra && (e = hipMemsetAsync(slot->d + align16(bytes.size()), 0, extra, stream)) != hipSuccess)
        return hip_status(fn, e);
    st->pending = true;
    st->seq = now;
    slot->bytes = bytes;
    slot->extra = extra;
    slot->last_use = now;
    d_plan = slot->d;
    return WQ_OK;
}

wq_status capture_state(const char* fn, hipStream_t stream, bool& capturing) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    const hipError_t e = hipStreamIsCapturing(stream, &cs);
    if (e != hipSuccess) return hip_status(fn, e);
    if (cs == hipStreamCaptureStatusInvalidated)
        return fail(WQ_ERR_HIP, "%s: the stream's capture has been invalidated", fn);
    capturing = cs == hipStreamCaptureStatusActive;
    return WQ_OK;
}

// One launch per dependency group (per batch chunk for M > 1), all on `stream`.
wq_status decode_grouped(const char* fn, const wq_linear* lin, int64_t count, int64_t m, hipStream_t stream) {
    std::vector<Group> groups;
    {
        wq::plan::SpanSet reads, writes;
        wq::plan::split_groups(lin, (int)count, m, reads, writes, [&](const Group& g) { groups.push_back(g); });
    }
    bool capturing = false;
    wq_status st = capture_state(fn, stream, capturing);
    if (st != WQ_OK) return st;
    std::lock_guard<std::mutex> guard(g_ws_mu);
    DecodeWorkspace* ws = nullptr;
    if ((st = get_workspace(fn, stream, ws)) != WQ_OK) return st;
    const bool matrix = wq::use_matrix_cores(m);
    std::vector<unsigned char> bytes(
        wq::plan::plan_bytes_bound(count, std::max(ws->shape.blocks4, ws->shape.blocks8)));
    PlanBuf pb{bytes.data(), bytes.size(), 0, false};
    std::vector<GroupPlan> gplans(groups.size());
    std::vector<BatchPlan> bplans(groups.size());
    const int64_t target = ws->shape.mb_waves[m <= 2 ? 0 : m <= 4 ? 1 : 2];
    for (size_t i = 0; i < groups.size(); ++i) {
        if (!groups[i].grouped) continue;
        if (m == 1) gplans[i] = wq::plan::plan_group(lin, groups[i], ws->shape.blocks4, ws->shape.blocks8, pb);
        else if (matrix) bplans[i] = wq::plan::plan_batch_group(lin, groups[i], pb);
        else bplans[i] = wq::plan::plan_vector_group(lin, groups[i], target, pb);
    }
    if (pb.overflow) return fail(WQ_ERR_INVALID_ARG, "%s: internal plan bound exceeded", fn);
    bytes.resize(pb.size);
    const unsigned char* d_plan = nullptr;
    if (!bytes.empty() && (st = place_plan(fn, ws, bytes, stream, capturing, d_plan)) != WQ_OK) return st;
    return hip_status(fn, wq::plan::launch_groups(lin, groups.data(), (int)groups.size(), gplans.data(),
                                                  bplans.data(), d_plan, m, matrix, stream));
}
}  // namespace

wq_status wq::record_error(wq_status st, const char* message) { return fail(st, "%s", message); }

wq_status wq::hip_error(const char* fn, hipError_t e) { return hip_status(fn, e); }

wq_status wq::resident_plan(const char* fn, hipStream_t stream, const std::vector<unsigned char>& bytes, size_t extra,
                            const unsigned char*& d_plan, size_t& extra_off, bool& capturing) {
    capturing = false;
    extra_off = align16(bytes.size());
    wq_status st = capture_state(fn, stream, capturing);
    if (st != WQ_OK) return st;
    std::lock_guard<std::mutex> guard(g_ws_mu);
    DecodeWorkspace* ws = nullptr;
    if ((st = get_workspace(fn, stream, ws)) != WQ_OK) return st;
    return place_plan(fn, ws, bytes, stream, capturing, d_plan, extra);
}

wq_status wq::check_decode_list(const char* fn, const wq_linear* lin, int64_t count, int64_t m, int64_t group,
                                wq::plan::Span* weights) {
    for (int64_t i = 0; i < count; ++i) {
        const wq_linear& l = lin[i];
        const GemvArgs a{l.packed_w, l.scales, l.x, l.y, l.N, l.K};
        const wq_status st = check_gemv(fn, a, m, group);
        if (st != WQ_OK) {
            char msg[512];
            snprintf(msg, sizeof(msg), "linear %lld: %s", (long long)i, g_last_error);
            return fail(st, "%s", msg);
        }
        weights[2 * i] = span_of(l.packed_w, l.N * l.K / 2);
        weights[2 * i + 1] = span_of(l.scales, l.N * (l.K / 32) * 2);
    }
    // No y may overlap any linear's weights: sort the weight spans, merge in
    // place, and binary-search each y.
    wq::plan::Span* end = weights + 2 * count;
    std::sort(weights, end, [](const Span& a, const Span& b) { return a.lo < b.lo; });
    int64_t merged = 0;
    for (wq::plan::Span* s = weights; s != end; ++s) {
        if (merged > 0 && s->lo <= weights[merged - 1].hi) weights[merged - 1].hi = std::max(weights[merged - 1].hi, s->hi);
        else weights[merged++] = *s;
    }
    for (int64_t i = 0; i < count; ++i) {
        const Span y = span_of(lin[i].y, 2 * m * lin[i].N);
        // First merged span starting at or after y.hi; only its predecessor
        // (the span with the largest start below y.hi) can overlap y.
        const wq::plan::Span* it = std::lower_bound(weights, weights + merged, y.hi,
                                                    [](const Span& s, uintptr_t v) { return s.lo < v; });
        if (it != weights && overlaps(*(it - 1), y))
            return fail(WQ_ERR_INVALID_ARG, "%s: y of linear %lld overlaps packed_w or scales of a linear", fn, (long long)i);
    }
    return WQ_OK;
}

extern "C" {

const char* wq_status_string(int status) {
    switch (status) {
        case WQ_OK: return "WQ_OK";
        case WQ_ERR_INVALID_ARG: return "WQ_ERR_INVALID_ARG";
        case WQ_ERR_UNSUPPORTED: return "WQ_ERR_UNSUPPORTED";
        case WQ_ERR_MISALIGNED: return "WQ_ERR_MISALIGNED";
        case WQ_ERR_HIP: return "WQ_ERR_HIP";
        default: return "WQ_UNKNOWN_STATUS";
    }
}

const char* wq_last_error_message(void) { return g_last_error; }

int wq_version(void) { return 100; }

wq_status wq_pack(const float* w, uint32_t* packed_w, uint16_t* scales, int64_t N, int64_t K,
                  int64_t group, void* stream) {
    static const char* fn = "wq_pack";
    if (!w || !packed_w || !scales) return fail(WQ_ERR_INVALID_ARG, "%s: null pointer", fn);
    wq_status st = check_shape(fn, N, K, group);
    if (st != WQ_OK) return st;
    if (!aligned(w, 16)) return fail(WQ_ERR_MISALIGNED, "%s: w must be 16-byte aligned", fn);
    if (!aligned(packed_w, 16)) return fail(WQ_ERR_MISALIGNED, "%s: packed_w must be 16-byte aligned", fn);
    if (!aligned(scales, 2)) return fail(WQ_ERR_MISALIGNED, "%s: scales must be 2-byte aligned", fn);
    const Span sw = span_of(w, 4 * N * K), sp = span_of(packed_w, N * K / 2), ss = span_of(scales, N * (K / 32) * 2);
    if (overlaps(sw, sp) || overlaps(sw, ss) || overlaps(sp, ss))
        return fail(WQ_ERR_INVALID_ARG, "%s: w, packed_w and scales must not overlap", fn);
    (void)hipGetLastError();
    return hip_status(fn, wq::launch_pack(w, packed_w, scales, N, K, static_cast<hipStream_t>(stream)));
}

wq_status wq_gemv(const uint32_t* packed_w, const uint16_t* scales, const uint16_t* x, uint16_t* y,
                  int64_t N, int64_t K, int64_t M, int64_t group, void* stream) {
    static const char* fn = "wq_gemv";
    const GemvArgs a{packed_w, scales, x, y, N, K};
    const wq_status st = check_gemv(fn, a, M, group);
    if (st != WQ_OK) return st;
    (void)hipGetLastError();
    return hip_status(fn, wq::launch_gemv(packed_w, scales, x, y, N, K, M, static_cast<hipStream_t>(stream)));
}

wq_status wq_decode_linears(const wq_linear* linears, int64_t count, int64_t M, int64_t group,
                            void* stream) {
    static const char* fn = "wq_decode_linears";
    if (!linears) return fail(WQ_ERR_INVALID_ARG, "%s: null descriptor array", fn);
    if (count <= 0 || count > WQ_MAX_LINEARS)
        return fail(WQ_ERR_INVALID_ARG, "%s: count must be in [1, %lld] (count=%lld)", fn, (long long)WQ_MAX_LINEARS, (long long)count);
    std::vector<wq::plan::Span> weights(2 * count);
    const wq_status st = wq::check_decode_list(fn, linears, count, M, group, weights.data());
    if (st != WQ_OK) return st;
    (void)hipGetLastError();
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (M <= wq::kMaxSmallBatchM) return decode_grouped(fn, linears, count, M, s);
    // Larger batches: one launch per linear, in stream order.
    for (int64_t i = 0; i < count; ++i) {
        const wq_linear& l = linears[i];
        const wq_status r = hip_status(fn, wq::launch_gemv(l.packed_w, l.scales, l.x, l.y, l.N, l.K, M, s));
        if (r != WQ_OK) return r;
    }
    return WQ_OK;
}

}  // extern "C"
