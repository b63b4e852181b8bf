// C ABI of the 4-bit decode-linear library: argument validation (entirely on
// the host, before any HIP call), kernel dispatch, and error reporting.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <utility>
#include <vector>

#include "wq.h"
#include "wq_internal.h"

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

struct Span {
    uintptr_t lo, hi;  // [lo, hi)
};

Span span_of(const void* p, int64_t bytes) {
    const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return Span{lo, lo + static_cast<uintptr_t>(bytes)};
}

bool overlaps(Span a, Span b) { return a.lo < b.hi && b.lo < a.hi; }

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
//
// Per (device, stream) workspace of the persistent decode kernel: the device
// copy of the linear table, the counter words, and a pinned staging buffer
// for table uploads.  Allocated on first use and kept until the process ends.
struct DecodeWorkspace {
    wq::DecodeEntry* d_table = nullptr;
    uint32_t* d_sync = nullptr;
    int capacity = 0;
    wq::DecodeEntry* h_stage = nullptr;
    hipEvent_t staged = nullptr;  // the last upload has been read by the device
    bool stage_pending = false;
    std::vector<wq::DecodeEntry> uploaded;
    uint32_t spin_limit = 1u << 18;  // polls of a dependency counter before giving up
    int blocks = 0;
};

std::mutex g_ws_mu;
std::map<std::pair<int, hipStream_t>, DecodeWorkspace*> g_ws;

// Target weight bytes per claimed tile: large for linears nothing waits on
// (a wave drains its pipeline when it moves to another linear), small where
// a dependency chain needs many waves on the same linear.
constexpr int64_t kTileBytesFree = 96 * 1024;
constexpr int64_t kTileBytesChained = 24 * 1024;

int rows_per_step(int gpl) { return gpl >= 8 ? 1 : 8 / gpl; }

// Build the kernel's view of the linears: tiling, dependencies, signals.
bool plan_decode(const std::vector<wq_linear>& lin, std::vector<wq::DecodeEntry>& ents, int& total_tiles,
                 int& max_gpl) {
    const int count = (int)lin.size();
    ents.assign(count, wq::DecodeEntry{});
    max_gpl = 1;
    for (int i = 0; i < count; ++i) {
        wq::DecodeEntry& e = ents[i];
        const wq_linear& l = lin[i];
        e.packed = l.packed_w;
        e.scales = l.scales;
        e.x = l.x;
        e.y = l.y;
        e.n = l.N;
        e.ng = (int32_t)(l.K / 32);
        e.gpl = (e.ng + 63) / 64;
        max_gpl = std::max(max_gpl, (int)e.gpl);
        e.dep0 = e.dep1 = -1;
        e.signal = 0;
    }
    // Linear i must wait for every earlier linear j whose output it reads,
    // whose input it overwrites, or whose output it overwrites.
    bool chain = count > 4096;
    for (int i = 0; i < count && !chain; ++i) {
        const Span xi = span_of(lin[i].x, 2 * lin[i].K), yi = span_of(lin[i].y, 2 * lin[i].N);
        int found = 0;
        for (int j = i - 1; j >= 0; --j) {
            const Span xj = span_of(lin[j].x, 2 * lin[j].K), yj = span_of(lin[j].y, 2 * lin[j].N);
            if (overlaps(xi, yj) || overlaps(yi, xj) || overlaps(yi, yj)) {
                if (found == 0) ents[i].dep0 = j;
                else if (found == 1) ents[i].dep1 = j;
                else chain = true;
                ++found;
            }
        }
    }
    if (chain) {
        // More than two conflicts somewhere: order every linear after its
        // predecessor, which orders it after all earlier ones.
        for (int i = 0; i < count; ++i) {
            ents[i].dep0 = i - 1;
            ents[i].dep1 = -1;
        }
    }
    for (int i = 0; i < count; ++i) {
        if (ents[i].dep0 >= 0) ents[ents[i].dep0].signal = 1;
        if (ents[i].dep1 >= 0) ents[ents[i].dep1].signal = 1;
    }
    int64_t tiles_total = 0;
    for (int i = 0; i < count; ++i) {
        wq::DecodeEntry& e = ents[i];
        const int64_t k = (int64_t)e.ng * 32;
        const int u = rows_per_step(e.gpl);
        const int64_t step_bytes = (int64_t)u * (k / 2 + 2 * e.ng);
        const bool chained = e.signal || e.dep0 >= 0 || e.dep1 >= 0;
        const int64_t target = chained ? kTileBytesChained : kTileBytesFree;
        const int64_t steps = std::max<int64_t>(1, (target + step_bytes / 2) / step_bytes);
        const int64_t rows = std::min<int64_t>(steps * u, ((e.n + u - 1) / u) * u);
        e.tile_rows = (int32_t)rows;
        e.tiles = (int32_t)((e.n + rows - 1) / rows);
        e.first_tile = (int32_t)tiles_total;
        tiles_total += e.tiles;
        if (tiles_total > 0x7fffffff) return false;
    }
    total_tiles = (int)tiles_total;
    return true;
}

wq_status get_workspace(const char* fn, hipStream_t stream, int count, DecodeWorkspace*& out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(fn, e);
    DecodeWorkspace*& ws = g_ws[std::make_pair(dev, stream)];
    if (!ws) {
        ws = new DecodeWorkspace();
        int cus = 0;
        if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
            return hip_status(fn, e);
        ws->blocks = std::max(1, cus) * 2;  // 8 waves per CU
        if (const char* env = std::getenv("WQ_DECODE_SPIN_LIMIT")) ws->spin_limit = (uint32_t)std::strtoul(env, nullptr, 10);
        if ((e = hipEventCreateWithFlags(&ws->staged, hipEventDisableTiming)) != hipSuccess) return hip_status(fn, e);
    }
    if (count > ws->capacity) {
        // Growing: make sure no launch still uses the old buffers.
        if (ws->d_table || ws->stage_pending) {
            if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_status(fn, e);
            ws->stage_pending = false;
        }
        if (ws->d_table) (void)hipFree(ws->d_table);
        if (ws->d_sync) (void)hipFree(ws->d_sync);
        if (ws->h_stage) (void)hipHostFree(ws->h_stage);
        ws->d_table = nullptr;
        ws->d_sync = nullptr;
        ws->h_stage = nullptr;
        ws->uploaded.clear();
        int cap = 64;
        while (cap < count) cap *= 2;
        if ((e = hipMalloc(reinterpret_cast<void**>(&ws->d_table), sizeof(wq::DecodeEntry) * cap)) != hipSuccess)
            return hip_status(fn, e);
        if ((e = hipMalloc(reinterpret_cast<void**>(&ws->d_sync), sizeof(uint32_t) * (wq::kSyncHeader + cap))) != hipSuccess)
            return hip_status(fn, e);
        if ((e = hipMemset(ws->d_sync, 0, sizeof(uint32_t) * (wq::kSyncHeader + cap))) != hipSuccess)
            return hip_status(fn, e);
        if ((e = hipHostMalloc(reinterpret_cast<void**>(&ws->h_stage), sizeof(wq::DecodeEntry) * cap)) != hipSuccess)
            return hip_status(fn, e);
        ws->capacity = cap;
    }
    out = ws;
    return WQ_OK;
}

// Run the linears with the persistent kernel (M = 1, K <= 16384).
wq_status decode_persistent(const char* fn, const std::vector<wq_linear>& lin, hipStream_t stream) {
    std::vector<wq::DecodeEntry> ents;
    int total_tiles = 0, max_gpl = 1;
    if (!plan_decode(lin, ents, total_tiles, max_gpl)) {
        for (const wq_linear& l : lin) {
            const wq_status st = hip_status(fn, wq::launch_gemv(l.packed_w, l.scales, l.x, l.y, l.N, l.K, 1, stream));
            if (st != WQ_OK) return st;
        }
        return WQ_OK;
    }
    const int count = (int)lin.size();
    std::lock_guard<std::mutex> guard(g_ws_mu);
    DecodeWorkspace* ws = nullptr;
    wq_status st = get_workspace(fn, stream, count, ws);
    if (st != WQ_OK) return st;
    hipError_t e;
    const size_t bytes = sizeof(wq::DecodeEntry) * count;
    if (ws->uploaded.size() != ents.size() || std::memcmp(ws->uploaded.data(), ents.data(), bytes) != 0) {
        if (ws->stage_pending && (e = hipEventSynchronize(ws->staged)) != hipSuccess) return hip_status(fn, e);
        std::memcpy(ws->h_stage, ents.data(), bytes);
        if ((e = hipMemcpyAsync(ws->d_table, ws->h_stage, bytes, hipMemcpyHostToDevice, stream)) != hipSuccess)
            return hip_status(fn, e);
        if ((e = hipEventRecord(ws->staged, stream)) != hipSuccess) return hip_status(fn, e);
        ws->stage_pending = true;
        ws->uploaded = ents;
    }
    return hip_status(fn, wq::launch_decode_m1(ws->d_table, count, total_tiles, max_gpl, ws->d_sync,
                                               ws->spin_limit, ws->blocks, stream));
}
}  // namespace

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
    std::vector<wq_linear> lin(linears, linears + count);
    std::vector<Span> weights;
    weights.reserve(2 * count);
    for (int64_t i = 0; i < count; ++i) {
        const wq_linear& l = lin[i];
        const GemvArgs a{l.packed_w, l.scales, l.x, l.y, l.N, l.K};
        const wq_status st = check_gemv(fn, a, M, group);
        if (st != WQ_OK) {
            char msg[512];
            snprintf(msg, sizeof(msg), "linear %lld: %s", (long long)i, g_last_error);
            return fail(st, "%s", msg);
        }
        weights.push_back(span_of(l.packed_w, l.N * l.K / 2));
        weights.push_back(span_of(l.scales, l.N * (l.K / 32) * 2));
    }
    // No y may overlap any linear's weights: sort the weight spans, merge, and
    // binary-search each y.
    std::sort(weights.begin(), weights.end(), [](const Span& a, const Span& b) { return a.lo < b.lo; });
    std::vector<Span> merged;
    for (const Span& s : weights) {
        if (!merged.empty() && s.lo <= merged.back().hi) merged.back().hi = std::max(merged.back().hi, s.hi);
        else merged.push_back(s);
    }
    for (int64_t i = 0; i < count; ++i) {
        const Span y = span_of(lin[i].y, 2 * M * lin[i].N);
        // First merged span starting at or after y.hi; only its predecessor
        // (the span with the largest start below y.hi) can overlap y.
        auto it = std::lower_bound(merged.begin(), merged.end(), y.hi, [](const Span& s, uintptr_t v) { return s.lo < v; });
        if (it != merged.begin() && overlaps(*std::prev(it), y)) return fail(WQ_ERR_INVALID_ARG, "%s: y of linear %lld overlaps packed_w or scales of a linear", fn, (long long)i);
    }
    (void)hipGetLastError();
    const hipStream_t s = static_cast<hipStream_t>(stream);
    bool persistent = (M == 1);
    for (int64_t i = 0; i < count && persistent; ++i)
        persistent = (lin[i].K / 32 + 63) / 64 <= wq::kDecodeMaxGpl && lin[i].N <= 0x7fffffff;
    if (persistent) return decode_persistent(fn, lin, s);
    // Other shapes: one launch per linear, in stream order.
    for (int64_t i = 0; i < count; ++i) {
        const wq_linear& l = lin[i];
        const wq_status st = hip_status(fn, wq::launch_gemv(l.packed_w, l.scales, l.x, l.y, l.N, l.K, M, s));
        if (st != WQ_OK) return st;
    }
    return WQ_OK;
}

}  // extern "C"
