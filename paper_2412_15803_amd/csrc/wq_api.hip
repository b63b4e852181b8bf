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

// A union of address intervals, kept merged, for the dependency checks.
class SpanSet {
  public:
    bool hits(Span s) const {
        if (s.lo >= s.hi) return false;
        auto it = m_.lower_bound(s.hi);  // first interval starting at or after s.hi
        if (it == m_.begin()) return false;
        --it;                            // the interval with the largest start below s.hi
        return it->second > s.lo;
    }
    void add(Span s) {
        if (s.lo >= s.hi) return;
        auto it = m_.upper_bound(s.lo);
        if (it != m_.begin() && std::prev(it)->second >= s.lo) {
            --it;
            s.lo = it->first;
            s.hi = std::max(s.hi, it->second);
            it = m_.erase(it);
        }
        while (it != m_.end() && it->first <= s.hi) {
            s.hi = std::max(s.hi, it->second);
            it = m_.erase(it);
        }
        m_[s.lo] = s.hi;
    }
    void clear() { m_.clear(); }

  private:
    std::map<uintptr_t, uintptr_t> m_;  // lo -> hi
};

// Split the linears into consecutive groups in which no linear reads the
// output of, or writes the input or output of, another linear of the same
// group.  Groups run in stream order, so this reproduces running the linears
// one after another.  Linears the grouped kernel cannot take (K > 16384, or
// codes of 4 GiB or more) form groups of their own.
struct Group {
    int begin, end;  // linear indices [begin, end)
    bool grouped;    // run with the grouped kernel (else one GEMV launch)
};

std::vector<Group> split_groups(const std::vector<wq_linear>& lin, int64_t m) {
    std::vector<Group> groups;
    SpanSet reads, writes;
    const int count = (int)lin.size();
    int begin = 0;
    for (int i = 0; i < count; ++i) {
        const wq_linear& l = lin[i];
        const bool too_long = m == 1 && l.K / 32 > 64 * wq::kDecodeMaxGpl;
        if (too_long || !wq::dev::fits_rsrc(l.N, l.K / 32)) {
            if (i > begin) groups.push_back(Group{begin, i, true});
            groups.push_back(Group{i, i + 1, false});
            reads.clear();
            writes.clear();
            begin = i + 1;
            continue;
        }
        const Span x = span_of(l.x, 2 * m * l.K), y = span_of(l.y, 2 * m * l.N);
        if (i > begin && (writes.hits(x) || reads.hits(y) || writes.hits(y))) {
            groups.push_back(Group{begin, i, true});
            reads.clear();
            writes.clear();
            begin = i;
        }
        reads.add(x);
        writes.add(y);
    }
    if (begin < count) groups.push_back(Group{begin, count, true});
    return groups;
}

int rows_per_step(int lpr, int gpl) { return wq::dev::step_rows_per_slot(gpl) * (64 / lpr); }

size_t align16(size_t v) { return (v + 15) & ~size_t(15); }

// Serialised plan of one grouped launch: [entries][classes][class list].
struct GroupPlan {
    size_t off_entries, off_classes, off_list;
    int nclasses;
    int max_gpl;
    int waves;
};

// Append the plan of linears [g.begin, g.end) to `bytes`.  `capacity` is
// the number of waves the device holds at once; classes get waves in
// proportion to their bytes, at least one and at most one per step.
GroupPlan plan_group(const std::vector<wq_linear>& lin, const Group& g, int capacity4, int capacity8,
                     std::vector<unsigned char>& bytes) {
    const int count = g.end - g.begin;
    std::vector<wq::DecodeEntry> ents(count, wq::DecodeEntry{});
    std::vector<wq::DecodeClass> cls;
    std::vector<std::vector<int32_t>> members;
    std::vector<double> work;
    int max_gpl = 1;
    for (int i = 0; i < count; ++i) {
        const wq_linear& l = lin[g.begin + i];
        wq::DecodeEntry& e = ents[i];
        e.packed = l.packed_w;
        e.scales = l.scales;
        e.x = l.x;
        e.y = l.y;
        e.n = l.N;
        e.ng = (int32_t)(l.K / 32);
        int lpr = 64, gpl = 1;
        wq::dev::pick_shape(e.ng, lpr, gpl);
        e.lpr = lpr;
        e.gpl = gpl;
        max_gpl = std::max(max_gpl, gpl);
        int ci = 0;
        while (ci < (int)cls.size() && !(cls[ci].lpr == lpr && cls[ci].gpl == gpl)) ++ci;
        if (ci == (int)cls.size()) {
            wq::DecodeClass c{};
            c.lpr = lpr;
            c.gpl = gpl;
            cls.push_back(c);
            members.emplace_back();
            work.push_back(0.0);
        }
        const int r = rows_per_step(lpr, gpl);
        e.steps = (e.n + r - 1) / r;
        e.first_step = cls[ci].steps;
        cls[ci].steps += e.steps;
        members[ci].push_back(i);
        work[ci] += (double)l.N * (double)(l.K / 2 + l.K / 16);
    }
    const int capacity = max_gpl <= 4 ? capacity4 : capacity8;
    double total = 0.0;
    for (double w : work) total += w;
    int waves = 0, off = 0;
    for (size_t c = 0; c < cls.size(); ++c) {
        int64_t wc = (int64_t)(capacity * work[c] / total);
        wc = std::max<int64_t>(1, std::min<int64_t>(wc, cls[c].steps));
        // A wave stages at most kYRows rows of y: at most that many rows' worth
        // of steps per wave, even if the class then gets more waves than its
        // share of the device.
        const int64_t max_steps = wq::dev::kYRows / rows_per_step(cls[c].lpr, cls[c].gpl);
        wc = std::max<int64_t>(wc, (cls[c].steps + max_steps - 1) / max_steps);
        cls[c].waves_begin = waves;
        cls[c].waves = (int32_t)wc;
        waves += (int)wc;
        cls[c].first = off;
        cls[c].count = (int32_t)members[c].size();
        off += cls[c].count;
    }
    GroupPlan gp;
    gp.nclasses = (int)cls.size();
    gp.max_gpl = max_gpl;
    gp.waves = waves;
    gp.off_entries = align16(bytes.size());
    gp.off_classes = align16(gp.off_entries + sizeof(wq::DecodeEntry) * count);
    gp.off_list = align16(gp.off_classes + sizeof(wq::DecodeClass) * cls.size());
    bytes.resize(align16(gp.off_list + sizeof(int32_t) * count), 0);
    std::memcpy(bytes.data() + gp.off_entries, ents.data(), sizeof(wq::DecodeEntry) * count);
    std::memcpy(bytes.data() + gp.off_classes, cls.data(), sizeof(wq::DecodeClass) * cls.size());
    int32_t* list = reinterpret_cast<int32_t*>(bytes.data() + gp.off_list);
    for (size_t c = 0; c < cls.size(); ++c)
        for (size_t m = 0; m < members[c].size(); ++m) list[cls[c].first + m] = members[c][m];
    return gp;
}

// Per (device, stream) workspace: the device copy of the last plan, a pinned
// staging buffer for uploads, and the device's resident-wave capacity.
// Allocated on first use and kept until the process ends.
struct DecodeWorkspace {
    unsigned char* d_plan = nullptr;
    unsigned char* h_stage = nullptr;
    size_t capacity = 0;                 // bytes of d_plan and h_stage
    hipEvent_t staged = nullptr;         // the last upload has been read by the device
    bool stage_pending = false;
    std::vector<unsigned char> uploaded; // bytes of the plan now in d_plan
    int waves4 = 0, waves8 = 0;          // resident waves of the two kernel variants
    int64_t mb_waves[3] = {0, 0, 0};     // target waves of the vector small-batch kernel, m <= 2, 4, 8
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
        if ((e = hipEventCreateWithFlags(&fresh->staged, hipEventDisableTiming)) != hipSuccess) return hip_status(fn, e);
        if ((e = wq::grouped_capacity(4, device, fresh->waves4)) != hipSuccess) return hip_status(fn, e);
        if ((e = wq::grouped_capacity(8, device, fresh->waves8)) != hipSuccess) return hip_status(fn, e);
        for (int i = 0; i < 3; ++i)
            if ((e = wq::mb_target_waves(2 << i, device, fresh->mb_waves[i])) != hipSuccess) return hip_status(fn, e);
        // Tuning override: fewer waves than the device holds (never more,
        // since every wave owns a fixed share of the work).
        if (const char* env = std::getenv("WQ_GROUPED_WAVES")) {
            const int w = std::atoi(env);
            if (w > 0) {
                fresh->waves4 = std::min(fresh->waves4, w);
                fresh->waves8 = std::min(fresh->waves8, w);
            }
        }
        // Tuning override: the vector small-batch kernel's target wave count.
        if (const char* env = std::getenv("WQ_MB_WAVES")) {
            const long long w = std::atoll(env);
            if (w > 0)
                for (int64_t& v : fresh->mb_waves) v = w;
        }
        ws = fresh.release();
    }
    out = ws;
    return WQ_OK;
}

// Make sure d_plan holds `bytes` (uploading only when it changed).
wq_status upload_plan(const char* fn, DecodeWorkspace* ws, std::vector<unsigned char>& bytes, hipStream_t stream) {
    if (ws->uploaded == bytes) return WQ_OK;
    hipError_t e;
    if (bytes.size() > ws->capacity) {
        // Growing: make sure no launch or copy still uses the old buffers.
        if (ws->d_plan && (e = hipStreamSynchronize(stream)) != hipSuccess) return hip_status(fn, e);
        if (ws->d_plan) (void)hipFree(ws->d_plan);
        if (ws->h_stage) (void)hipHostFree(ws->h_stage);
        ws->d_plan = nullptr;
        ws->h_stage = nullptr;
        ws->stage_pending = false;
        ws->uploaded.clear();
        size_t cap = 4096;
        while (cap < bytes.size()) cap *= 2;
        if ((e = hipMalloc(reinterpret_cast<void**>(&ws->d_plan), cap)) != hipSuccess) return hip_status(fn, e);
        if ((e = hipHostMalloc(reinterpret_cast<void**>(&ws->h_stage), cap)) != hipSuccess) return hip_status(fn, e);
        ws->capacity = cap;
    }
    if (ws->stage_pending && (e = hipEventSynchronize(ws->staged)) != hipSuccess) return hip_status(fn, e);
    std::memcpy(ws->h_stage, bytes.data(), bytes.size());
    if ((e = hipMemcpyAsync(ws->d_plan, ws->h_stage, bytes.size(), hipMemcpyHostToDevice, stream)) != hipSuccess)
        return hip_status(fn, e);
    if ((e = hipEventRecord(ws->staged, stream)) != hipSuccess) return hip_status(fn, e);
    ws->stage_pending = true;
    ws->uploaded.swap(bytes);
    return WQ_OK;
}

wq_status decode_per_linear(const char* fn, const wq_linear* lin, int64_t count, int64_t m, hipStream_t stream) {
    for (int64_t i = 0; i < count; ++i) {
        const wq_linear& l = lin[i];
        const wq_status st = hip_status(fn, wq::launch_gemv(l.packed_w, l.scales, l.x, l.y, l.N, l.K, m, stream));
        if (st != WQ_OK) return st;
    }
    return WQ_OK;
}

// M = 1: one grouped launch per dependency group (one GEMV launch for the
// linears the grouped kernel cannot take), all on `stream`.
wq_status decode_grouped(const char* fn, const std::vector<wq_linear>& lin, hipStream_t stream) {
    const std::vector<Group> groups = split_groups(lin, 1);
    std::lock_guard<std::mutex> guard(g_ws_mu);
    DecodeWorkspace* ws = nullptr;
    wq_status st = get_workspace(fn, stream, ws);
    if (st != WQ_OK) return st;
    std::vector<unsigned char> bytes;
    std::vector<GroupPlan> plans(groups.size());
    for (size_t i = 0; i < groups.size(); ++i)
        if (groups[i].grouped) plans[i] = plan_group(lin, groups[i], ws->waves4, ws->waves8, bytes);
    if (!bytes.empty() && (st = upload_plan(fn, ws, bytes, stream)) != WQ_OK) return st;
    for (size_t i = 0; i < groups.size(); ++i) {
        const Group& g = groups[i];
        if (!g.grouped) {
            if ((st = decode_per_linear(fn, &lin[g.begin], g.end - g.begin, 1, stream)) != WQ_OK) return st;
            continue;
        }
        const GroupPlan& gp = plans[i];
        wq::DecodePlan p;
        p.entries = reinterpret_cast<const wq::DecodeEntry*>(ws->d_plan + gp.off_entries);
        p.classes = reinterpret_cast<const wq::DecodeClass*>(ws->d_plan + gp.off_classes);
        p.class_lin = reinterpret_cast<const int32_t*>(ws->d_plan + gp.off_list);
        p.nclasses = gp.nclasses;
        if ((st = hip_status(fn, wq::launch_grouped_m1(p, gp.max_gpl, gp.waves, stream))) != WQ_OK) return st;
    }
    return WQ_OK;
}
// Plan of one small-batch grouped launch: the entries, each owning a run of
// blocks (tiles of grouped_mfma_tiles() x 16 rows) of the grid.
struct BatchPlan {
    size_t off_entries;
    int count;
    int64_t blocks;
    int waves_per_block;
};

BatchPlan plan_batch_group(const std::vector<wq_linear>& lin, const Group& g, std::vector<unsigned char>& bytes) {
    const int count = g.end - g.begin;
    const int rows_per_block = 16 * wq::grouped_mfma_tiles();
    std::vector<wq::DecodeEntry> ents(count, wq::DecodeEntry{});
    int64_t blocks = 0, max_steps = 1;
    for (int i = 0; i < count; ++i) {
        const wq_linear& l = lin[g.begin + i];
        wq::DecodeEntry& e = ents[i];
        e.packed = l.packed_w;
        e.scales = l.scales;
        e.x = l.x;
        e.y = l.y;
        e.n = l.N;
        e.ng = (int32_t)(l.K / 32);
        e.first_step = blocks;
        e.steps = (l.N + rows_per_block - 1) / rows_per_block;
        blocks += e.steps;
        max_steps = std::max<int64_t>(max_steps, (e.ng + 3) / 4);
    }
    BatchPlan bp;
    bp.count = count;
    bp.blocks = blocks;
    // About 32 steps of the longest row per wave (measured on the 3B- and
    // 8B-class steps: fewer, longer waves keep more blocks resident per CU).
    bp.waves_per_block = (int)std::min<int64_t>(8, (max_steps + 31) / 32);
    bp.off_entries = align16(bytes.size());
    bytes.resize(align16(bp.off_entries + sizeof(wq::DecodeEntry) * count), 0);
    std::memcpy(bytes.data() + bp.off_entries, ents.data(), sizeof(wq::DecodeEntry) * count);
    return bp;
}

// 2 <= M < 8 on the vector ALUs: one launch per dependency group and 8
// batch rows; waves own row runs of one linear each.  The runs are sized so
// that every wave streams about the same number of (row, padded group)
// pairs, `target` waves in all (fixed-size runs would give a K = 8192 wave
// 2.7 times the work of a K = 3072 one, and the CUs holding those waves
// would set the time).
BatchPlan plan_vector_group(const std::vector<wq_linear>& lin, const Group& g, int64_t target,
                            std::vector<unsigned char>& bytes) {
    const int count = g.end - g.begin;
    int64_t work = 0;
    for (int i = 0; i < count; ++i) work += lin[g.begin + i].N * wq::mb_padded_groups(lin[g.begin + i].K / 32);
    const int64_t per_wave = (work + target - 1) / target;
    std::vector<wq::DecodeEntry> ents(count, wq::DecodeEntry{});
    int64_t waves = 0;
    for (int i = 0; i < count; ++i) {
        const wq_linear& l = lin[g.begin + i];
        wq::DecodeEntry& e = ents[i];
        e.packed = l.packed_w;
        e.scales = l.scales;
        e.x = l.x;
        e.y = l.y;
        e.n = l.N;
        e.ng = (int32_t)(l.K / 32);
        e.pad = wq::mb_rows_for_work(per_wave, e.ng);
        e.first_step = waves;
        e.steps = (l.N + e.pad - 1) / e.pad;
        waves += e.steps;
    }
    BatchPlan bp;
    bp.count = count;
    bp.blocks = waves;  // waves, for this plan
    bp.waves_per_block = 0;
    bp.off_entries = align16(bytes.size());
    bytes.resize(align16(bp.off_entries + sizeof(wq::DecodeEntry) * count), 0);
    std::memcpy(bytes.data() + bp.off_entries, ents.data(), sizeof(wq::DecodeEntry) * count);
    return bp;
}

// M >= 2: one matrix-core launch per dependency group and 16 batch rows
// (from kMatrixCoreMinM rows on), else one vector launch per group and 8.
wq_status decode_grouped_batch(const char* fn, const std::vector<wq_linear>& lin, int64_t m, hipStream_t stream) {
    const std::vector<Group> groups = split_groups(lin, m);
    std::lock_guard<std::mutex> guard(g_ws_mu);
    DecodeWorkspace* ws = nullptr;
    wq_status st = get_workspace(fn, stream, ws);
    if (st != WQ_OK) return st;
    std::vector<unsigned char> bytes;
    const bool matrix = m >= wq::kMatrixCoreMinM && !wq::vector_small_batch();
    std::vector<BatchPlan> plans(groups.size());
    for (size_t i = 0; i < groups.size(); ++i)
        if (groups[i].grouped)
            plans[i] = matrix ? plan_batch_group(lin, groups[i], bytes)
                              : plan_vector_group(lin, groups[i], ws->mb_waves[m <= 2 ? 0 : m <= 4 ? 1 : 2], bytes);
    if (!bytes.empty() && (st = upload_plan(fn, ws, bytes, stream)) != WQ_OK) return st;
    for (size_t i = 0; i < groups.size(); ++i) {
        const Group& g = groups[i];
        if (!g.grouped) {
            if ((st = decode_per_linear(fn, &lin[g.begin], g.end - g.begin, m, stream)) != WQ_OK) return st;
            continue;
        }
        const BatchPlan& bp = plans[i];
        const wq::DecodeEntry* ents = reinterpret_cast<const wq::DecodeEntry*>(ws->d_plan + bp.off_entries);
        const int64_t chunk = matrix ? 16 : 8;
        for (int64_t m0 = 0; m0 < m; m0 += chunk) {
            const int mc = (int)std::min<int64_t>(chunk, m - m0);
            st = hip_status(fn, matrix ? wq::launch_grouped_mfma(ents, bp.count, bp.blocks, bp.waves_per_block, m0, mc, stream)
                                       : wq::launch_grouped_mb(ents, bp.count, bp.blocks, m0, mc, stream));
            if (st != WQ_OK) return st;
        }
    }
    return WQ_OK;
}
}  // namespace

wq_status wq::record_error(wq_status st, const char* message) { return fail(st, "%s", message); }

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
    if (M == 1) return decode_grouped(fn, lin, s);
    if (M <= 64) return decode_grouped_batch(fn, lin, M, s);
    // Larger batches: one launch per linear, in stream order.
    return decode_per_linear(fn, lin.data(), count, M, s);
}

}  // extern "C"
