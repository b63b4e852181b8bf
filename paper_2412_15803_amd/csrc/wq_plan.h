// Host-side planning of a decode step (wq_decode_linears and its
// no-allocation variant): dependency grouping of the descriptor list and the
// serialised per-launch plans the grouped kernels read.  Nothing here
// allocates: plans are written into a caller-provided byte buffer, and the
// dependency sets are supplied by the caller (a std::map-backed set for long
// lists, a fixed array for the no-allocation path).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <map>
#include <vector>

#include "wq.h"
#include "wq_internal.h"

namespace wq {
namespace plan {

struct Span {
    uintptr_t lo, hi;  // [lo, hi)
};

inline Span span_of(const void* p, int64_t bytes) {
    const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return Span{lo, lo + static_cast<uintptr_t>(bytes)};
}

inline bool overlaps(Span a, Span b) { return a.lo < b.hi && b.lo < a.hi; }

// A union of address intervals, kept merged (any number of spans).
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

// The same interface over caller-owned storage of `cap` spans, searched
// linearly (the no-allocation path, whose lists are short).
class SpanList {
  public:
    SpanList(Span* store, int cap) : s_(store), cap_(cap) {}
    bool hits(Span s) const {
        for (int i = 0; i < n_; ++i)
            if (overlaps(s_[i], s)) return true;
        return false;
    }
    void add(Span s) {
        if (s.lo < s.hi && n_ < cap_) s_[n_++] = s;
    }
    void clear() { n_ = 0; }

  private:
    Span* s_;
    int cap_;
    int n_ = 0;
};

// Consecutive linears [begin, end) that run in one launch.
struct Group {
    int begin, end;
    bool grouped;  // run with a grouped kernel (else one GEMV launch per linear)
};

// Rows of one group at most: the grouped kernels number a launch's steps
// (at most one per row) in 32-bit integers.
constexpr int64_t kGroupMaxRows = int64_t(1) << 30;

// Split linears[0, count) into consecutive groups in which no linear reads the
// output of, or writes the input or output of, another linear of the same
// group.  Groups run in stream order, so this reproduces running the linears
// one after another.  Linears the grouped kernels cannot take (K > 16384 at
// M = 1, or codes of 4 GiB or more) form groups of their own, and a group
// closes before its rows would pass kGroupMaxRows.  Calls emit(Group) in
// order; `reads` and `writes` are empty dependency sets.
template <class Deps, class Emit>
void split_groups(const wq_linear* lin, int count, int64_t m, Deps& reads, Deps& writes, Emit emit) {
    int begin = 0;
    int64_t rows = 0;
    for (int i = 0; i < count; ++i) {
        const wq_linear& l = lin[i];
        const bool too_long = m == 1 && l.K / 32 > 64 * kDecodeMaxGpl;
        if (too_long || !fits_rsrc(l.N, l.K / 32)) {
            if (i > begin) emit(Group{begin, i, true});
            emit(Group{i, i + 1, false});
            reads.clear();
            writes.clear();
            begin = i + 1;
            rows = 0;
            continue;
        }
        const Span x = span_of(l.x, 2 * m * l.K), y = span_of(l.y, 2 * m * l.N);
        if (i > begin && (writes.hits(x) || reads.hits(y) || writes.hits(y) || rows + l.N > kGroupMaxRows)) {
            emit(Group{begin, i, true});
            reads.clear();
            writes.clear();
            begin = i;
            rows = 0;
        }
        reads.add(x);
        writes.add(y);
        rows += l.N;
    }
    if (begin < count) emit(Group{begin, count, true});
}

// A byte buffer the plans are appended to; `overflow` is set (and nothing
// written) when a plan does not fit.
struct PlanBuf {
    unsigned char* data;
    size_t cap;
    size_t size;
    bool overflow;
};

// Bytes of the plans of `count` linears in any grouping, for sizing a
// PlanBuf: per group at most entries + classes + class list + the shares of
// at most `max_blocks` + kMaxClasses workgroups, each 16-byte aligned.
inline size_t plan_bytes_bound(int64_t count, int max_blocks) {
    return (size_t)count * (sizeof(DecodeEntry) + sizeof(int32_t) + 80 + sizeof(DecodeClass) * kMaxClasses +
                            sizeof(DecodeBlock) * ((size_t)max_blocks + kMaxClasses));
}

// Plan of one batch-1 grouped launch: offsets into the plan bytes.
struct GroupPlan {
    size_t off_entries, off_classes, off_list, off_blocks;
    int nclasses;
    int max_gpl;
    int blocks;
};

// Plan of one small-batch grouped launch: entries, each owning a run of
// blocks (matrix cores) or waves (vector kernel) of the grid.
struct BatchPlan {
    size_t off_entries;
    int count;
    int64_t blocks;
    int waves_per_block;
};

// Append the batch-1 plan of linears [g.begin, g.end); `capacity4` and
// `capacity8` are the workgroups the device holds at once of the narrow and
// wide grouped kernels.
GroupPlan plan_group(const wq_linear* lin, const Group& g, int capacity4, int capacity8, PlanBuf& out);

// Append the matrix-core (M >= 3) plan of a group.
BatchPlan plan_batch_group(const wq_linear* lin, const Group& g, PlanBuf& out);

// Append the vector small-batch (M < 8) plan of a group, `target` waves.
BatchPlan plan_vector_group(const wq_linear* lin, const Group& g, int64_t target, PlanBuf& out);

// The device's resident-wave capacities the planners need.
struct DeviceShape {
    int blocks4 = 0, blocks8 = 0;     // grouped batch-1 kernel, narrow and wide variants
    int64_t mb_waves[3] = {0, 0, 0};  // vector small-batch target waves for m <= 2, 4, 8
};

// Query `device` (hipOccupancy* and attributes, no allocation) and apply the
// WQ_GROUPED_BLOCKS and WQ_MB_WAVES tuning overrides.
hipError_t device_shape(int device, DeviceShape& out);

// Launch one call's planned groups in order on `stream`.  `d_plan` is the
// device address of the plan bytes; groups[i] uses gplans[i] (M = 1) or
// bplans[i] (M > 1); ungrouped groups run one wq_gemv launch per linear.
// `matrix` tells the batch path which kernel its plans were made for.
hipError_t launch_groups(const wq_linear* lin, const Group* groups, int ngroups, const GroupPlan* gplans,
                         const BatchPlan* bplans, const unsigned char* d_plan, int64_t m, bool matrix,
                         hipStream_t stream);

}  // namespace plan

// Place `bytes` in one of the library-owned plan buffers of the current
// device and `stream` (the resident plans wq_decode_linears keeps, see
// include/wq.h) and return its device address: no copy when the same bytes
// are resident already.  `extra` more bytes of device memory follow the plan
// at offset `extra_off` (16-byte aligned); they are zeroed when the plan is
// uploaded and otherwise left as the device last wrote them (state that
// belongs to this plan).  Under stream capture only a resident plan is
// accepted, and its buffer is frozen; otherwise WQ_ERR_UNSUPPORTED is
// returned and nothing is recorded.  `capturing` reports the stream's state.
wq_status resident_plan(const char* fn, hipStream_t stream, const std::vector<unsigned char>& bytes, size_t extra,
                        const unsigned char*& d_plan, size_t& extra_off, bool& capturing);

// Validation shared by the decode-step entry points (defined with the C ABI):
// every descriptor as for wq_gemv, and no y overlapping any linear's codes or
// scales.  `weights` is caller storage for 2 * count spans.  On failure the
// thread's error message names the entry point `fn` and the linear.
wq_status check_decode_list(const char* fn, const wq_linear* lin, int64_t count, int64_t m, int64_t group,
                            plan::Span* weights);

}  // namespace wq
