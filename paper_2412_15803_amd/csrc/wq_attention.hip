// Decode-step attention over a paged KV cache (gfx950, wave64): the attention
// of one new token per sequence over the keys and values that the engine
// keeps in a paged cache (Sec. 2.2), computed the way PagedAttention-style
// kernels do (Sec. 2.3): scores, softmax and the weighted sum of values in
// one pass over the cache, split along the sequence where one workgroup per
// head would leave the chip idle.
//
// Work split.  A sequence is cut into chunks of T tokens (a multiple of 64).  One
// 256-thread workgroup takes one (sequence, kv head, chunk) and serves all G
// query heads of that kv head, so every cached key and value is read from HBM
// once.  Each of its four waves takes a contiguous quarter of the chunk.
//
// Lane layout.  A wave-wide 16-byte load covers four tokens: lanes
// 16r .. 16r + 15 (row r) hold dims 8c .. 8c + 7 (c = lane % 16) of token r,
// 256 contiguous bytes per token.  A "block" is four such loads of keys and
// four of values (16 tokens of one wave); blocks are double-buffered in
// registers.  Scores are 16-lane DPP sums of v_dot2 partials (exact fp16
// products, fp32 sums) and end up in every lane of the row.  Each row keeps a
// running softmax state per query head: the maximum m of its scores (in
// log2 units), l = sum 2^(a - m) and acc = sum 2^(a - m) V over its 8 dims,
// rescaled once per block.
//
// Merging.  The four row states of a wave are merged across lanes with
// v_permlane16/32_swap exchanges, the four wave states through LDS.  With
// one chunk per sequence the workgroup then writes the fp16 output;
// otherwise it writes (m, l, acc) to the workspace and merge_kernel combines
// the chunks of every (sequence, query head) in a second launch.  When the
// (sequence, kv head) pairs divide evenly over the XCDs, all chunks of a pair
// and the merge of its heads run on one XCD, so the merge finds the partial
// results in that XCD's L2.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>

#include "wq_attention.h"
#include "wq_device.h"
#include "wq_internal.h"

namespace wq {
namespace attn {
namespace {

using dev::as_h2;
using dev::gbl;
using dev::half2v;
using dev::u32x4;

constexpr int kD = WQ_ATTN_HEAD_DIM;
constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kRowsPerLoad = 4;                              // tokens per wave-wide load
constexpr int kLoadsPerBlock = 4;
constexpr int kBlockTokens = kRowsPerLoad * kLoadsPerBlock;  // 16 tokens of one wave
constexpr int kChunkQuantum = kWaves * kBlockTokens;        // 64 tokens: a block per wave
constexpr int kMaxChunk = 4096;
constexpr int kMaxSplits = 1024;
static_assert(WQ_ATTN_MAX_SEQ_LEN / kMaxChunk <= kMaxSplits, "chunks per sequence stay bounded");
constexpr uint16_t kHalfNaN = 0x7E00;
// Workgroups of a launch are dealt to the XCDs in turn (workgroup b runs on
// XCD b % kXcds), and each XCD has its own L2.
constexpr int kXcds = 8;

static_assert(kD == 128, "the lane layout assumes 16 lanes x 8 dims per token");

struct Params {
    const uint16_t* q;
    const uint16_t* k;
    const uint16_t* v;
    const int32_t* table;
    const int32_t* lens;
    uint16_t* out;
    float* part_acc;    // [seq * hq + h][splits][kD]
    float2* part_ml;    // [seq * hq + h][splits]: (m, l)
    int64_t max_pages;  // row length of the block table
    uint32_t page_stride;  // elements per page: hkv * page_size * kD
    int32_t num_pages;
    int32_t hq, hkv;
    int32_t log2_page;
    int32_t chunk;            // tokens per chunk, a multiple of kChunkQuantum
    int32_t splits;
    int32_t max_seq_len;
    int32_t pages_per_chunk;  // block-table entries one chunk can use
    int32_t pages_lds;        // bytes of LDS before the wave states
    int32_t xcd_local;        // nonzero: pairs are placed by XCD (xcd_pair)
    float c;            // scale * log2(e): scores in log2 units
};

__device__ __forceinline__ bool bad_length(const Params& p, int len) {
    return len < 0 || len > p.max_seq_len || (int64_t)len > (p.max_pages << p.log2_page);
}

__device__ __forceinline__ uint16_t to_half_bits(float x) {
    return __builtin_bit_cast(uint16_t, static_cast<_Float16>(x));
}

__device__ __forceinline__ float exp2_(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float dot8(const half2v (&q)[4], const u32x4 k) {
    float a = __builtin_amdgcn_fdot2(q[0], as_h2(k.x), 0.0f, false);
    a = __builtin_amdgcn_fdot2(q[1], as_h2(k.y), a, false);
    a = __builtin_amdgcn_fdot2(q[2], as_h2(k.z), a, false);
    return __builtin_amdgcn_fdot2(q[3], as_h2(k.w), a, false);
}

__device__ __forceinline__ void unpack8(const u32x4 v, float (&f)[8]) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const half2v h = as_h2(w[i]);
        f[2 * i] = static_cast<float>(h.x);
        f[2 * i + 1] = static_cast<float>(h.y);
    }
}

struct KVBlock {
    u32x4 k[kLoadsPerBlock];
    u32x4 v[kLoadsPerBlock];
};

// Running softmax state of one query head in one lane (8 dims of a row).
struct State {
    float m, l, acc[8];
};

// Fold the states of the two lanes of a pair into one, the pair being lanes
// l and l ^ 16 (kHalves false) or l and l ^ 32 (kHalves true).
// v_permlane16_swap of a register with itself hands each lane the values of
// the even and odd 16-lane row of its pair, v_permlane32_swap those of the
// lower and upper 32 lanes, so both lanes merge the same two states in the
// same order (lower first) and end with the same bits.  Both are VALU
// exchanges: no LDS round trip per value.
template <bool kHalves>
__device__ __forceinline__ void pair_values(float x, float& lo, float& hi) {
    const uint32_t b = __builtin_bit_cast(uint32_t, x);
    uint32_t e0, e1;
    // (Non-const results: with `const auto` this compiler reads element 0
    // for both elements of the returned pair.)
    if constexpr (kHalves) {
        auto p = __builtin_amdgcn_permlane32_swap(b, b, false, false);
        e0 = p[0];
        e1 = p[1];
    } else {
        auto p = __builtin_amdgcn_permlane16_swap(b, b, false, false);
        e0 = p[0];
        e1 = p[1];
    }
    lo = __builtin_bit_cast(float, e0);
    hi = __builtin_bit_cast(float, e1);
}

template <bool kHalves>
__device__ __forceinline__ void fold_pair(State& st) {
    float m0, m1, l0, l1;
    pair_values<kHalves>(st.m, m0, m1);
    pair_values<kHalves>(st.l, l0, l1);
    const float mx = fmaxf(m0, m1);
    const float ms = mx == -INFINITY ? 0.0f : mx;
    const float w0 = exp2_(m0 - ms), w1 = exp2_(m1 - ms);
    st.l = fmaf(l1, w1, l0 * w0);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        float a0, a1;
        pair_values<kHalves>(st.acc[e], a0, a1);
        st.acc[e] = fmaf(a1, w1, a0 * w0);
    }
    st.m = mx;
}

template <int G>
__global__ __launch_bounds__(kThreads) void split_kernel(const Params p) {
    extern __shared__ __align__(16) unsigned char smem[];
    int* sh_pages = reinterpret_cast<int*>(smem);
    float* sh_acc = reinterpret_cast<float*>(smem + p.pages_lds);  // [kWaves][G][kD]
    float* sh_m = sh_acc + kWaves * G * kD;                           // [kWaves][G]
    float* sh_l = sh_m + kWaves * G;

    const int tid = threadIdx.x;
    // (sequence, kv head) pair and chunk of this workgroup.  With xcd_local
    // the pairs are dealt to the XCDs and every chunk of a pair runs on its
    // pair's XCD, as does the merge of its heads, so the merge reads the
    // partial results from that XCD's L2 instead of from memory.
    int chunk, seq_kv;
    if (p.xcd_local) {
        const int x = blockIdx.x % kXcds, i = blockIdx.x / kXcds;
        seq_kv = x + kXcds * (i / p.splits);
        chunk = i % p.splits;
    } else {
        chunk = blockIdx.x % p.splits;
        seq_kv = blockIdx.x / p.splits;
    }
    const int kvh = seq_kv % p.hkv;
    const int s = seq_kv / p.hkv;
    const int64_t head0 = (int64_t)s * p.hq + (int64_t)kvh * G;  // first query head of the group

    const int lane = tid & 63, row = lane >> 4, col = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int log2_page = p.log2_page;
    const int page_mask = (1 << log2_page) - 1;
    const int c0 = chunk * p.chunk;
    const int first_page = c0 >> log2_page;

    // One round trip for the length, the query vectors and the block-table
    // entries the chunk may use (bounded by the table row: the length is not
    // known yet).  Entries are checked against the cache size when used.
    const int len = p.lens[s];
    half2v qv[G][4];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const u32x4 t = *gbl(reinterpret_cast<const u32x4*>(p.q + (head0 + g) * kD + col * 8));
        qv[g][0] = as_h2(t.x);
        qv[g][1] = as_h2(t.y);
        qv[g][2] = as_h2(t.z);
        qv[g][3] = as_h2(t.w);
    }
    const int32_t* trow = p.table + (int64_t)s * p.max_pages + first_page;
    const int table_left = (int)min<int64_t>(p.pages_per_chunk, p.max_pages - first_page);
    for (int i = tid; i < table_left; i += kThreads) sh_pages[i] = trow[i];
    __syncthreads();

    if (bad_length(p, len) || len == 0) {
        if (p.splits == 1) {
            const uint16_t fill = len == 0 ? 0 : kHalfNaN;
            for (int i = tid; i < G * kD; i += kThreads) p.out[head0 * kD + i] = fill;
        }
        return;
    }
    if (c0 >= len) return;
    int bad = 0;

    // This wave's tokens: [wbase, wbase + wtok) intersected with [0, len).
    const int wtok = p.chunk / kWaves;
    const int wbase = c0 + wave * wtok;
    const int nvalid = min(max(len - wbase, 0), wtok);
    const int nblk = (nvalid + kBlockTokens - 1) / kBlockTokens;
    const uint32_t head_slot0 = (uint32_t)kvh << log2_page;

    // Loads of block `blk`.  Rows past the end of the sequence read its last
    // token again (already cached) so that every block issues the same loads.
    auto issue = [&](KVBlock& b, int blk) {
#pragma unroll
        for (int j = 0; j < kLoadsPerBlock; ++j) {
            const int t = min(wbase + blk * kBlockTokens + j * kRowsPerLoad + row, len - 1);
            uint32_t pg = (uint32_t)sh_pages[(t >> log2_page) - first_page];
            if (pg >= (uint32_t)p.num_pages) {
                bad = 1;
                pg = 0;
            }
            const uint64_t off = (uint64_t)pg * p.page_stride +
                                 (uint64_t)((head_slot0 + (uint32_t)(t & page_mask)) * kD + col * 8);
            // Non-temporal: every cached key and value is read once per call,
            // and streaming them past L2 keeps the block table, q and the
            // partial results there (6-11% faster on the measured shapes).
            b.k[j] = __builtin_nontemporal_load(gbl(reinterpret_cast<const u32x4*>(p.k + off)));
            b.v[j] = __builtin_nontemporal_load(gbl(reinterpret_cast<const u32x4*>(p.v + off)));
        }
    };

    State st[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
        st[g].m = -INFINITY;
        st[g].l = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) st[g].acc[e] = 0.0f;
    }

    auto compute = [&](const KVBlock& b, int blk) {
        float sc[G][kLoadsPerBlock];
#pragma unroll
        for (int j = 0; j < kLoadsPerBlock; ++j) {
            const bool ok = wbase + blk * kBlockTokens + j * kRowsPerLoad + row < len;
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const float d = dev::segment_sum<16>(dot8(qv[g], b.k[j]));
                sc[g][j] = ok ? d * p.c : -INFINITY;
            }
        }
        // Rescale each head's state to the block's new maximum and turn the
        // scores into weights, then add the weighted values slab by slab (only
        // one slab's values are unpacked at a time).
#pragma unroll
        for (int g = 0; g < G; ++g) {
            float mx = st[g].m;
#pragma unroll
            for (int j = 0; j < kLoadsPerBlock; ++j) mx = fmaxf(mx, sc[g][j]);
            const float ms = mx == -INFINITY ? 0.0f : mx;
            const float corr = exp2_(st[g].m - ms);
            float l = st[g].l * corr;
#pragma unroll
            for (int e = 0; e < 8; ++e) st[g].acc[e] *= corr;
#pragma unroll
            for (int j = 0; j < kLoadsPerBlock; ++j) {
                sc[g][j] = exp2_(sc[g][j] - ms);
                l += sc[g][j];
            }
            st[g].l = l;
            st[g].m = mx;
        }
#pragma unroll
        for (int j = 0; j < kLoadsPerBlock; ++j) {
            float vf[8];
            unpack8(b.v[j], vf);
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int e = 0; e < 8; ++e) st[g].acc[e] = fmaf(sc[g][j], vf[e], st[g].acc[e]);
        }
    };

    // Double-buffered: the next block's loads are in flight while a block is
    // computed.  Every path issues a buffer's loads before the other buffer's
    // compute, so the compiler's wait counts stay exact.
    if (nblk > 0) {
        KVBlock a, b;
        issue(a, 0);
        int blk = 0;
        bool last_in_a = true;
        while (blk + 1 < nblk) {
            issue(b, blk + 1);
            compute(a, blk);
            if (++blk + 1 >= nblk) {
                last_in_a = false;
                break;
            }
            issue(a, blk + 1);
            compute(b, blk);
            ++blk;
        }
        if (last_in_a) compute(a, blk);
        else compute(b, blk);
    }

    // Merge the four rows of the wave, then the four waves.
#pragma unroll
    for (int g = 0; g < G; ++g) {
        fold_pair<false>(st[g]);
        fold_pair<true>(st[g]);
    }
    // A wave that met a page number outside the cache stores a NaN sum, which
    // every later fold carries into the output (fmaf(NaN, w, .) is NaN for
    // any weight), so one plain barrier does instead of a reduction.
    const bool wave_bad = __builtin_amdgcn_ballot_w64(bad != 0) != 0;
    if (row == 0) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            float* dst = sh_acc + (wave * G + g) * kD + col * 8;
            *reinterpret_cast<float4*>(dst) = make_float4(st[g].acc[0], st[g].acc[1], st[g].acc[2], st[g].acc[3]);
            *reinterpret_cast<float4*>(dst + 4) = make_float4(st[g].acc[4], st[g].acc[5], st[g].acc[6], st[g].acc[7]);
            if (col == 0) {
                sh_m[wave * G + g] = st[g].m;
                sh_l[wave * G + g] = wave_bad ? NAN : st[g].l;
            }
        }
    }
    __syncthreads();
    for (int i = tid; i < G * kD; i += kThreads) {
        const int g = i / kD, d = i % kD;
        float mx = -INFINITY;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) mx = fmaxf(mx, sh_m[w * G + g]);
        float l = 0.0f, acc = 0.0f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const float wt = exp2_(sh_m[w * G + g] - mx);
            l = fmaf(sh_l[w * G + g], wt, l);
            acc = fmaf(sh_acc[(w * G + g) * kD + d], wt, acc);
        }
        if (p.splits == 1) {
            p.out[(head0 + g) * kD + d] = l != l ? kHalfNaN : to_half_bits(acc / l);
        } else {
            const int64_t slot = (head0 + g) * p.splits + chunk;
            p.part_acc[slot * kD + d] = acc;
            if (d == 0) p.part_ml[slot] = make_float2(mx, l);
        }
    }
}

// One workgroup per (sequence, query head): out = sum_c 2^(m_c - M) acc_c /
// sum_c 2^(m_c - M) l_c over the sequence's chunks, M = max_c m_c.  Thread
// (slot, col) folds chunks slot, slot + 8, ... of dims 4 col .. 4 col + 3
// into a running state; the first batch of chunk loads is issued together
// with the length (only chunks below the launch's split count, all inside
// the workspace), so short sequences take one round trip.  The eight slot
// states are then merged through LDS.
__global__ __launch_bounds__(kThreads) void merge_kernel(const Params p) {
    constexpr int kCols = kD / 4;             // 32 four-dim columns
    constexpr int kSlots = kThreads / kCols;  // 8 chunk slots
    constexpr int kBatch = 8;                 // chunks per slot loaded at once
    __shared__ float sh_m[kSlots], sh_l[kSlots];
    __shared__ float4 sh_a[kSlots][kCols];

    const int tid = threadIdx.x;
    const int slot = tid / kCols, cq = tid % kCols;
    int64_t head = blockIdx.x;  // seq * hq + h
    if (p.xcd_local) {  // the heads of pair x + 8 j run on XCD x
        const int group = p.hq / p.hkv;
        const int x = blockIdx.x % kXcds, i = blockIdx.x / kXcds;
        const int pair = x + kXcds * (i / group);
        head = (int64_t)(pair / p.hkv) * p.hq + (int64_t)(pair % p.hkv) * group + i % group;
    }
    const int s = (int)(head / p.hq);
    uint16_t* o = p.out + head * kD;
    const float2* ml = p.part_ml + head * p.splits;
    const float4* pa = reinterpret_cast<const float4*>(p.part_acc + head * p.splits * kD) + cq;

    const int len = p.lens[s];
    float m = -INFINITY, l = 0.0f;
    float4 a = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    int n = p.splits;  // chunks that hold data; known once the length arrives
    for (int base = slot; base < n; base += kSlots * kBatch) {
        float2 h[kBatch];
        float4 v[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            const int c = min(base + j * kSlots, p.splits - 1);
            h[j] = ml[c];
            v[j] = pa[(int64_t)c * kCols];
        }
        if (base == slot) {
            if (bad_length(p, len) || len == 0) break;
            n = (len + p.chunk - 1) / p.chunk;
        }
        float mx = m;
#pragma unroll
        for (int j = 0; j < kBatch; ++j)
            if (base + j * kSlots < n) mx = fmaxf(mx, h[j].x);
        if (mx == -INFINITY) break;  // no chunk of this slot holds data
        const float corr = exp2_(m - mx);
        l *= corr;
        a.x *= corr;
        a.y *= corr;
        a.z *= corr;
        a.w *= corr;
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            if (base + j * kSlots >= n) continue;
            const float w = exp2_(h[j].x - mx);
            l = fmaf(h[j].y, w, l);
            a.x = fmaf(w, v[j].x, a.x);
            a.y = fmaf(w, v[j].y, a.y);
            a.z = fmaf(w, v[j].z, a.z);
            a.w = fmaf(w, v[j].w, a.w);
        }
        m = mx;
    }
    if (bad_length(p, len) || len == 0) {
        if (tid < kD) o[tid] = len == 0 ? 0 : kHalfNaN;
        return;
    }
    if (cq == 0) {
        sh_m[slot] = m;
        sh_l[slot] = l;
    }
    sh_a[slot][cq] = a;
    __syncthreads();
    if (tid < kD) {
        float mx = -INFINITY;
#pragma unroll
        for (int sl = 0; sl < kSlots; ++sl) mx = fmaxf(mx, sh_m[sl]);
        const float* col = reinterpret_cast<const float*>(&sh_a[0][0]) + tid;
        float lt = 0.0f, acc = 0.0f;
#pragma unroll
        for (int sl = 0; sl < kSlots; ++sl) {
            const float w = exp2_(sh_m[sl] - mx);
            lt = fmaf(sh_l[sl], w, lt);
            acc = fmaf(col[sl * kD], w, acc);
        }
        o[tid] = to_half_bits(acc / lt);
    }
}

// ------------------------------------------------------------------- host

struct Plan {
    int64_t chunk;
    int64_t splits;
    size_t ml_offset;  // bytes of part_acc
    size_t ws_bytes;
};

bool xcd_placement() {
    const char* e = getenv("WQ_ATTN_XCD_LOCAL");
    return !e || strtol(e, nullptr, 10) != 0;
}

int64_t target_blocks() {
    const char* e = getenv("WQ_ATTN_TARGET_BLOCKS");
    const long v = e ? strtol(e, nullptr, 10) : 0;
    return v > 0 ? v : 512;
}

// Chunk length: a multiple of 64 tokens that gives the split launch about
// target_blocks() workgroups (what the chip holds at once, so there is a
// single round of them), at most kMaxChunk tokens; with sequences of at most
// WQ_ATTN_MAX_SEQ_LEN tokens that keeps a sequence within kMaxSplits chunks.
Plan make_plan(int64_t seqs, int64_t hq, int64_t hkv, int64_t max_seq_len) {
    const int64_t len = std::max<int64_t>(max_seq_len, 1);
    const int64_t want = std::max<int64_t>(1, target_blocks() / (seqs * hkv));  // chunks per sequence
    int64_t chunk = (len + want - 1) / want;
    chunk = (chunk + kChunkQuantum - 1) / kChunkQuantum * kChunkQuantum;
    chunk = std::min<int64_t>(std::max<int64_t>(chunk, kChunkQuantum), kMaxChunk);
    Plan pl{chunk, (len + chunk - 1) / chunk, 0, 0};
    if (pl.splits > 1) {
        pl.ml_offset = (size_t)(seqs * hq * pl.splits * kD * 4);
        pl.ws_bytes = pl.ml_offset + (size_t)(seqs * hq * pl.splits * 8);
    }
    return pl;
}

template <int G>
hipError_t launch_split(const Params& p, int64_t blocks, size_t lds, hipStream_t stream) {
    hipLaunchKernelGGL(split_kernel<G>, dim3((unsigned)blocks), dim3(kThreads), lds, stream, p);
    return hipGetLastError();
}

hipError_t launch(const Params& p, int group, int64_t seqs, hipStream_t stream) {
    const int64_t blocks = seqs * p.hkv * p.splits;
    const size_t lds = (size_t)p.pages_lds + (size_t)kWaves * group * (kD + 2) * 4;
    hipError_t e;
    switch (group) {
        case 1: e = launch_split<1>(p, blocks, lds, stream); break;
        case 2: e = launch_split<2>(p, blocks, lds, stream); break;
        case 3: e = launch_split<3>(p, blocks, lds, stream); break;
        case 4: e = launch_split<4>(p, blocks, lds, stream); break;
        case 5: e = launch_split<5>(p, blocks, lds, stream); break;
        case 6: e = launch_split<6>(p, blocks, lds, stream); break;
        case 7: e = launch_split<7>(p, blocks, lds, stream); break;
        default: e = launch_split<8>(p, blocks, lds, stream); break;
    }
    if (e != hipSuccess || p.splits == 1) return e;
    hipLaunchKernelGGL(merge_kernel, dim3((unsigned)(seqs * p.hq)), dim3(kThreads), 0, stream, p);
    return hipGetLastError();
}

wq_status err(wq_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
wq_status err(wq_status st, const char* fmt, ...) {
    char msg[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(msg, sizeof(msg), fmt, ap);
    va_end(ap);
    return record_error(st, msg);
}

bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }
int log2_of(int64_t v) {
    int r = 0;
    while ((int64_t(1) << r) < v) ++r;
    return r;
}
bool aligned(const void* ptr, uintptr_t a) { return reinterpret_cast<uintptr_t>(ptr) % a == 0; }

struct Span {
    uintptr_t lo, hi;
};
Span span(const void* ptr, uint64_t bytes) {
    const uintptr_t lo = reinterpret_cast<uintptr_t>(ptr);
    return Span{lo, lo + (uintptr_t)bytes};
}
bool overlaps(Span a, Span b) { return a.lo < a.hi && b.lo < b.hi && a.lo < b.hi && b.lo < a.hi; }

wq_status check_sizes(const char* fn, int64_t seqs, int64_t hq, int64_t hkv, int64_t head_dim,
                      int64_t max_seq_len) {
    if (seqs < 1 || seqs > WQ_ATTN_MAX_SEQS)
        return err(WQ_ERR_INVALID_ARG, "%s: num_seqs must be in [1, %lld] (got %lld)", fn,
                   (long long)WQ_ATTN_MAX_SEQS, (long long)seqs);
    if (hkv < 1 || hkv > WQ_ATTN_MAX_KV_HEADS)
        return err(WQ_ERR_INVALID_ARG, "%s: num_kv_heads must be in [1, %d] (got %lld)", fn,
                   WQ_ATTN_MAX_KV_HEADS, (long long)hkv);
    if (hq < 1 || hq % hkv != 0)
        return err(WQ_ERR_INVALID_ARG, "%s: num_q_heads (%lld) must be a positive multiple of num_kv_heads (%lld)",
                   fn, (long long)hq, (long long)hkv);
    if (hq / hkv > WQ_ATTN_MAX_GROUP)
        return err(WQ_ERR_UNSUPPORTED, "%s: at most %d query heads per kv head (got %lld)", fn,
                   WQ_ATTN_MAX_GROUP, (long long)(hq / hkv));
    if (head_dim != WQ_ATTN_HEAD_DIM)
        return err(WQ_ERR_UNSUPPORTED, "%s: head_dim must be %d (got %lld)", fn, WQ_ATTN_HEAD_DIM,
                   (long long)head_dim);
    if (max_seq_len < 0 || max_seq_len > WQ_ATTN_MAX_SEQ_LEN)
        return err(WQ_ERR_INVALID_ARG, "%s: max_seq_len must be in [0, %lld] (got %lld)", fn,
                   (long long)WQ_ATTN_MAX_SEQ_LEN, (long long)max_seq_len);
    const Plan pl = make_plan(seqs, hq, hkv, max_seq_len);
    if (seqs * hkv * pl.splits > INT32_MAX || seqs * hq > INT32_MAX)
        return err(WQ_ERR_INVALID_ARG, "%s: too many workgroups for one launch", fn);
    return WQ_OK;
}

}  // namespace
}  // namespace attn
}  // namespace wq

using namespace wq::attn;

extern "C" {

wq_status wq_paged_attention_workspace_size(int64_t num_seqs, int64_t num_q_heads, int64_t num_kv_heads,
                                            int64_t head_dim, int64_t max_seq_len, size_t* bytes) {
    static const char* fn = "wq_paged_attention_workspace_size";
    if (!bytes) return err(WQ_ERR_INVALID_ARG, "%s: null output pointer", fn);
    const wq_status st = check_sizes(fn, num_seqs, num_q_heads, num_kv_heads, head_dim, max_seq_len);
    if (st != WQ_OK) return st;
    *bytes = make_plan(num_seqs, num_q_heads, num_kv_heads, max_seq_len).ws_bytes;
    return WQ_OK;
}

wq_status wq_paged_attention(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                             const int32_t* block_table, const int32_t* seq_lens, uint16_t* out,
                             int64_t num_seqs, int64_t num_q_heads, int64_t num_kv_heads, int64_t head_dim,
                             int64_t page_size, int64_t num_pages, int64_t max_pages_per_seq,
                             int64_t max_seq_len, float scale, void* workspace, size_t workspace_bytes,
                             void* stream) {
    static const char* fn = "wq_paged_attention";
    if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !out)
        return err(WQ_ERR_INVALID_ARG, "%s: null pointer", fn);
    wq_status st = check_sizes(fn, num_seqs, num_q_heads, num_kv_heads, head_dim, max_seq_len);
    if (st != WQ_OK) return st;
    if (!is_pow2(page_size) || page_size > WQ_ATTN_MAX_PAGE_SIZE)
        return err(WQ_ERR_UNSUPPORTED, "%s: page_size must be a power of two in [1, %d] (got %lld)", fn,
                   WQ_ATTN_MAX_PAGE_SIZE, (long long)page_size);
    if (num_pages < 1 || num_pages > INT32_MAX)
        return err(WQ_ERR_INVALID_ARG, "%s: num_pages must be in [1, 2^31 - 1] (got %lld)", fn, (long long)num_pages);
    if (max_pages_per_seq < 1 || max_pages_per_seq > INT32_MAX)
        return err(WQ_ERR_INVALID_ARG, "%s: max_pages_per_seq must be in [1, 2^31 - 1] (got %lld)", fn,
                   (long long)max_pages_per_seq);
    if (max_seq_len > max_pages_per_seq * page_size)
        return err(WQ_ERR_INVALID_ARG, "%s: max_seq_len %lld exceeds max_pages_per_seq * page_size", fn,
                   (long long)max_seq_len);
    if (!std::isfinite(scale)) return err(WQ_ERR_INVALID_ARG, "%s: scale must be finite", fn);
    if (!aligned(q, 16) || !aligned(out, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16))
        return err(WQ_ERR_MISALIGNED, "%s: q, out, k_cache and v_cache must be 16-byte aligned", fn);
    if (!aligned(block_table, 4) || !aligned(seq_lens, 4))
        return err(WQ_ERR_MISALIGNED, "%s: block_table and seq_lens must be 4-byte aligned", fn);

    const Plan pl = make_plan(num_seqs, num_q_heads, num_kv_heads, max_seq_len);
    if (pl.ws_bytes > 0) {
        if (!workspace) return err(WQ_ERR_INVALID_ARG, "%s: a workspace of %zu bytes is needed", fn, pl.ws_bytes);
        if (workspace_bytes < pl.ws_bytes)
            return err(WQ_ERR_INVALID_ARG, "%s: workspace of %zu bytes is below the %zu needed", fn, workspace_bytes,
                       pl.ws_bytes);
        if (!aligned(workspace, 16)) return err(WQ_ERR_MISALIGNED, "%s: workspace must be 16-byte aligned", fn);
    }
    const uint64_t qo_bytes = (uint64_t)num_seqs * num_q_heads * head_dim * 2;
    const uint64_t cache_bytes = (uint64_t)num_pages * num_kv_heads * page_size * head_dim * 2;
    const Span so = span(out, qo_bytes);
    const Span sw = span(workspace, pl.ws_bytes);
    const Span inputs[] = {span(q, qo_bytes), span(k_cache, cache_bytes), span(v_cache, cache_bytes),
                           span(block_table, (uint64_t)num_seqs * max_pages_per_seq * 4),
                           span(seq_lens, (uint64_t)num_seqs * 4)};
    for (const Span& in : inputs) {
        if (overlaps(so, in)) return err(WQ_ERR_INVALID_ARG, "%s: out overlaps an input", fn);
        if (overlaps(sw, in)) return err(WQ_ERR_INVALID_ARG, "%s: the workspace overlaps an input", fn);
    }
    if (overlaps(so, sw)) return err(WQ_ERR_INVALID_ARG, "%s: out overlaps the workspace", fn);

    const int group = (int)(num_q_heads / num_kv_heads);
    const int log2_page = log2_of(page_size);
    // Pages a chunk can touch: it may start inside a page.
    const int64_t pages_per_chunk = (pl.chunk >> log2_page) + 2;

    Params p{};
    p.q = q;
    p.k = k_cache;
    p.v = v_cache;
    p.table = block_table;
    p.lens = seq_lens;
    p.out = out;
    p.part_acc = pl.ws_bytes ? static_cast<float*>(workspace) : nullptr;
    p.part_ml = pl.ws_bytes ? reinterpret_cast<float2*>(static_cast<char*>(workspace) + pl.ml_offset) : nullptr;
    p.max_pages = max_pages_per_seq;
    p.page_stride = (uint32_t)(num_kv_heads * page_size * head_dim);
    p.num_pages = (int32_t)num_pages;
    p.hq = (int32_t)num_q_heads;
    p.hkv = (int32_t)num_kv_heads;
    p.log2_page = log2_page;
    p.chunk = (int32_t)pl.chunk;
    p.splits = (int32_t)pl.splits;
    p.max_seq_len = (int32_t)max_seq_len;
    p.pages_per_chunk = (int32_t)pages_per_chunk;
    p.pages_lds = (int32_t)((pages_per_chunk * 4 + 15) / 16 * 16);
    p.c = (float)((double)scale * 1.4426950408889634);  // log2(e)
    // Place pairs by XCD only when every XCD gets the same number of them.
    p.xcd_local = pl.splits > 1 && (num_seqs * num_kv_heads) % kXcds == 0 && xcd_placement();

    (void)hipGetLastError();
    const hipError_t e = launch(p, group, num_seqs, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return err(WQ_ERR_HIP, "%s: HIP error %d (%s)", fn, (int)e, hipGetErrorString(e));
    return WQ_OK;
}

}  // extern "C"
