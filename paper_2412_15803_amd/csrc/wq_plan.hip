// Host-side planning of a decode step's grouped launches (see wq_plan.h).
// Plans are written into a caller-provided buffer; nothing here allocates.
#include <cstdlib>
#include <cstring>

#include "wq_device.h"
#include "wq_plan.h"

namespace wq {
namespace plan {

namespace {

size_t align16(size_t v) { return (v + 15) & ~size_t(15); }

// Rows per step of a batch-1 grouped launch whose widest linear has
// `max_gpl` groups of x per lane (the kernel variant it runs on).
int rows_per_step(int lpr, int gpl, int max_gpl) {
    return dev::step_rows_per_slot(gpl, dev::grouped_step_loads(max_gpl)) * (64 / lpr);
}

void fill_entry(DecodeEntry& e, const wq_linear& l) {
    e = DecodeEntry{};
    e.packed = l.packed_w;
    e.scales = l.scales;
    e.x = l.x;
    e.y = l.y;
    e.n = l.N;
    e.ng = (int32_t)(l.K / 32);
}

int class_of(const DecodeClass* cls, int ncls, int lpr, int gpl) {
    for (int c = 0; c < ncls; ++c)
        if (cls[c].lpr == lpr && cls[c].gpl == gpl) return c;
    return -1;
}

}  // namespace

// What a row costs beyond its bytes (its reduction and output), in bytes of
// streaming: measured on the 3B-class step, whose K = 3072 rows (1728 bytes)
// took about 8% longer per byte than its K = 8192 rows (4608 bytes) when
// workgroups were split by bytes alone.
constexpr double kRowCost = 256.0;

// Classes (linears of one step shape) get workgroups in proportion to their
// bytes plus kRowCost per row, at least one and at most one per step; every
// workgroup then streams one contiguous range of its class's steps.
GroupPlan plan_group(const wq_linear* lin, const Group& g, int capacity4, int capacity8, PlanBuf& out) {
    const int count = g.end - g.begin;
    GroupPlan gp{};
    DecodeClass cls[kMaxClasses] = {};
    double work[kMaxClasses] = {};
    int ncls = 0, max_gpl = 1;
    for (int i = 0; i < count; ++i) {
        int lpr = 64, gpl = 1;
        dev::pick_shape((int)(lin[g.begin + i].K / 32), lpr, gpl);
        max_gpl = std::max(max_gpl, gpl);
    }
    for (int i = 0; i < count; ++i) {
        const wq_linear& l = lin[g.begin + i];
        int lpr = 64, gpl = 1;
        dev::pick_shape((int)(l.K / 32), lpr, gpl);
        int c = class_of(cls, ncls, lpr, gpl);
        if (c < 0) {
            c = ncls++;  // pick_shape returns at most kMaxClasses distinct shapes
            cls[c].lpr = lpr;
            cls[c].gpl = gpl;
        }
        const int r = rows_per_step(lpr, gpl, max_gpl);
        cls[c].steps += (l.N + r - 1) / r;
        cls[c].count += 1;
        work[c] += (double)l.N * ((double)(l.K / 2 + l.K / 16) + kRowCost);
    }
    gp.nclasses = ncls;
    gp.max_gpl = max_gpl;
    gp.off_entries = align16(out.size);
    gp.off_classes = align16(gp.off_entries + sizeof(DecodeEntry) * count);
    gp.off_list = align16(gp.off_classes + sizeof(DecodeClass) * ncls);
    const int capacity = max_gpl <= 4 ? capacity4 : capacity8;
    double total = 0.0;
    for (int c = 0; c < ncls; ++c) total += work[c];
    int blocks = 0, off = 0;
    for (int c = 0; c < ncls; ++c) {
        int64_t bc = (int64_t)(capacity * work[c] / total);
        bc = std::max<int64_t>(1, std::min<int64_t>(bc, cls[c].steps));
        cls[c].blocks_begin = blocks;
        cls[c].blocks = (int32_t)bc;
        blocks += (int)bc;
        cls[c].first = off;
        off += cls[c].count;
    }
    gp.off_blocks = align16(gp.off_list + sizeof(int32_t) * count);
    const size_t end = align16(gp.off_blocks + sizeof(DecodeBlock) * blocks);
    if (out.overflow || end > out.cap) {
        out.overflow = true;
        return gp;
    }
    std::memset(out.data + out.size, 0, end - out.size);
    DecodeEntry* ents = reinterpret_cast<DecodeEntry*>(out.data + gp.off_entries);
    int32_t* list = reinterpret_cast<int32_t*>(out.data + gp.off_list);
    // Entries in list order, each with its first step in its class's
    // numbering; the class lists name the linears of a class in order.
    int64_t next_step[kMaxClasses] = {};
    int filled[kMaxClasses] = {};
    for (int i = 0; i < count; ++i) {
        const wq_linear& l = lin[g.begin + i];
        DecodeEntry& e = ents[i];
        fill_entry(e, l);
        int lpr = 64, gpl = 1;
        dev::pick_shape(e.ng, lpr, gpl);
        e.lpr = lpr;
        e.gpl = gpl;
        const int c = class_of(cls, ncls, lpr, gpl);
        const int r = rows_per_step(lpr, gpl, max_gpl);
        e.steps = (e.n + r - 1) / r;
        e.first_step = next_step[c];
        next_step[c] += e.steps;
        list[cls[c].first + filled[c]++] = i;
    }
    // Per workgroup, its equal share of its class's steps and the list
    // position of the linear holding the share's first step (the workgroups
    // of a class start at increasing steps).
    DecodeBlock* blk = reinterpret_cast<DecodeBlock*>(out.data + gp.off_blocks);
    for (int c = 0; c < ncls; ++c) {
        int k = 0;
        for (int j = 0; j < cls[c].blocks; ++j) {
            const int64_t first = (int64_t)j * cls[c].steps / cls[c].blocks;
            while (k + 1 < cls[c].count) {
                const DecodeEntry& e = ents[list[cls[c].first + k]];
                if (first < e.first_step + e.steps) break;
                ++k;
            }
            DecodeBlock& b = blk[cls[c].blocks_begin + j];
            b.pos = k;
            b.begin = (int32_t)first;
            b.end = (int32_t)((int64_t)(j + 1) * cls[c].steps / cls[c].blocks);
        }
    }
    std::memcpy(out.data + gp.off_classes, cls, sizeof(DecodeClass) * ncls);
    gp.blocks = blocks;
    out.size = end;
    return gp;
}

#ifndef WQ_MFMA_WAVE_STEPS
#define WQ_MFMA_WAVE_STEPS 32
#endif
constexpr int64_t kMfmaWaveSteps = WQ_MFMA_WAVE_STEPS;

BatchPlan plan_batch_group(const wq_linear* lin, const Group& g, PlanBuf& out) {
    const int count = g.end - g.begin;
    const int rows_per_block = 16 * grouped_mfma_tiles();
    BatchPlan bp{};
    bp.count = count;
    bp.off_entries = align16(out.size);
    const size_t end = align16(bp.off_entries + sizeof(DecodeEntry) * count);
    if (out.overflow || end > out.cap) {
        out.overflow = true;
        return bp;
    }
    std::memset(out.data + out.size, 0, end - out.size);
    DecodeEntry* ents = reinterpret_cast<DecodeEntry*>(out.data + bp.off_entries);
    int64_t blocks = 0, max_steps = 1;
    for (int i = 0; i < count; ++i) {
        const wq_linear& l = lin[g.begin + i];
        DecodeEntry& e = ents[i];
        fill_entry(e, l);
        e.first_step = blocks;
        e.steps = (l.N + rows_per_block - 1) / rows_per_block;
        blocks += e.steps;
        max_steps = std::max<int64_t>(max_steps, (e.ng + 3) / 4);
    }
    bp.blocks = blocks;
    // About 32 steps of the longest row per wave (measured on the 3B- and
    // 8B-class steps: fewer, longer waves keep more blocks resident per CU),
    // at most 4 (each wave's scale-window slots take 16 KiB of LDS).
    bp.waves_per_block = (int)std::min<int64_t>(grouped_mfma_max_waves(), (max_steps + kMfmaWaveSteps - 1) / kMfmaWaveSteps);
    out.size = end;
    return bp;
}

// Row runs sized so that every wave streams about the same number of (row,
// padded group) pairs, `target` waves in all (fixed-size runs would give a
// K = 8192 wave 2.7 times the work of a K = 3072 one, and the CUs holding
// those waves would set the time).
BatchPlan plan_vector_group(const wq_linear* lin, const Group& g, int64_t target, PlanBuf& out) {
    const int count = g.end - g.begin;
    BatchPlan bp{};
    bp.count = count;
    bp.waves_per_block = 0;
    bp.off_entries = align16(out.size);
    const size_t end = align16(bp.off_entries + sizeof(DecodeEntry) * count);
    if (out.overflow || end > out.cap) {
        out.overflow = true;
        return bp;
    }
    std::memset(out.data + out.size, 0, end - out.size);
    int64_t work = 0;
    for (int i = 0; i < count; ++i) work += lin[g.begin + i].N * mb_padded_groups(lin[g.begin + i].K / 32);
    const int64_t per_wave = (work + target - 1) / target;
    DecodeEntry* ents = reinterpret_cast<DecodeEntry*>(out.data + bp.off_entries);
    int64_t waves = 0;
    for (int i = 0; i < count; ++i) {
        const wq_linear& l = lin[g.begin + i];
        DecodeEntry& e = ents[i];
        fill_entry(e, l);
        e.pad = mb_rows_for_work(per_wave, e.ng);
        e.first_step = waves;
        e.steps = (l.N + e.pad - 1) / e.pad;
        waves += e.steps;
    }
    bp.blocks = waves;  // waves, for this plan
    out.size = end;
    return bp;
}

hipError_t device_shape(int device, DeviceShape& out) {
    hipError_t e;
    if ((e = grouped_capacity(4, device, out.blocks4)) != hipSuccess) return e;
    if ((e = grouped_capacity(8, device, out.blocks8)) != hipSuccess) return e;
    for (int i = 0; i < 3; ++i)
        if ((e = mb_target_waves(2 << i, device, out.mb_waves[i])) != hipSuccess) return e;
    // Tuning override: fewer workgroups than the device holds (never more,
    // since every workgroup owns a fixed share of the work).
    if (const char* env = std::getenv("WQ_GROUPED_BLOCKS")) {
        const int b = std::atoi(env);
        if (b > 0) {
            out.blocks4 = std::min(out.blocks4, b);
            out.blocks8 = std::min(out.blocks8, b);
        }
    }
    // Tuning override: the vector small-batch kernel's target wave count.
    if (const char* env = std::getenv("WQ_MB_WAVES")) {
        const long long w = std::atoll(env);
        if (w > 0)
            for (int64_t& v : out.mb_waves) v = w;
    }
    return hipSuccess;
}

hipError_t launch_groups(const wq_linear* lin, const Group* groups, int ngroups, const GroupPlan* gplans,
                         const BatchPlan* bplans, const unsigned char* d_plan, int64_t m, bool matrix,
                         hipStream_t stream) {
    for (int i = 0; i < ngroups; ++i) {
        const Group& g = groups[i];
        hipError_t e = hipSuccess;
        if (!g.grouped) {
            for (int j = g.begin; j < g.end && e == hipSuccess; ++j)
                e = launch_gemv(lin[j].packed_w, lin[j].scales, lin[j].x, lin[j].y, lin[j].N, lin[j].K, m, stream);
        } else if (m == 1) {
            const GroupPlan& gp = gplans[i];
            DecodePlan p;
            p.entries = reinterpret_cast<const DecodeEntry*>(d_plan + gp.off_entries);
            p.classes = reinterpret_cast<const DecodeClass*>(d_plan + gp.off_classes);
            p.class_lin = reinterpret_cast<const int32_t*>(d_plan + gp.off_list);
            p.blocks = reinterpret_cast<const DecodeBlock*>(d_plan + gp.off_blocks);
            p.nclasses = gp.nclasses;
            e = launch_grouped_m1(p, gp.max_gpl, gp.blocks, stream);
        } else {
            const BatchPlan& bp = bplans[i];
            const DecodeEntry* ents = reinterpret_cast<const DecodeEntry*>(d_plan + bp.off_entries);
            const int64_t chunk = matrix ? 16 : 8;
            for (int64_t m0 = 0; m0 < m && e == hipSuccess; m0 += chunk) {
                const int mc = (int)std::min<int64_t>(chunk, m - m0);
                e = matrix ? launch_grouped_mfma(ents, bp.count, bp.blocks, bp.waves_per_block, m0, mc, stream)
                           : launch_grouped_mb(ents, bp.count, bp.blocks, m0, mc, stream);
            }
        }
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace plan
}  // namespace wq
