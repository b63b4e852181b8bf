// C ABI of the 4-bit decode-linear library: argument validation (entirely on
// the host, before any HIP call), kernel dispatch, and error reporting.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
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
    for (int64_t i = 0; i < count; ++i) {
        const wq_linear& l = lin[i];
        const wq_status st = hip_status(fn, wq::launch_gemv(l.packed_w, l.scales, l.x, l.y, l.N, l.K, M, s));
        if (st != WQ_OK) return st;
    }
    return WQ_OK;
}

}  // extern "C"
