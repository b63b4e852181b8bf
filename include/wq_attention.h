/*
 * wq_attention.h -- C ABI of decode-step attention over a paged KV cache, in
 * the same library as wq.h (libwq.so; status codes and error messages are
 * shared with it).
 *
 * The operation is the attention of one decoding step (Sec. 2.2: the engine
 * keeps every sequence's keys and values in a paged KV cache; Sec. 2.3:
 * PagedAttention-style kernels compute attention over that cache).  For each
 * sequence s (one new query token) and query head h:
 *
 *     a_t     = scale * sum_d q[s][h][d] * K_t[d]          0 <= t < L_s
 *     o[s][h] = sum_t softmax(a)_t * V_t
 *
 * where K_t / V_t are the cached key / value vectors of token t of sequence s
 * for kv head h / G (G = num_q_heads / num_kv_heads, grouped-query heads).
 * An empty sequence (L_s = 0) has the zero vector as output.
 *
 * Cache layout (this library's choice; the paper fixes none):
 *   k_cache, v_cache  [num_pages][num_kv_heads][page_size][head_dim] IEEE
 *                     binary16, row-major.  Token t of sequence s is slot
 *                     t % page_size of page block_table[s][t / page_size].
 *   block_table       [num_seqs][max_pages_per_seq] int32.  Only entries
 *                     below ceil(L_s / page_size) are read.
 *   seq_lens          [num_seqs] int32, L_s.
 *   q, out            [num_seqs][num_q_heads][head_dim] binary16.
 * Every pointer is a DEVICE pointer owned by the caller; the library keeps
 * none of them after the call.  Calls are asynchronous and stream-ordered.
 *
 * Numerics: scores, softmax and the weighted sum are computed in fp32; each
 * output is rounded once to fp16.  Per element the result is within
 * 2e-3 * sum_t w_t |V_t[d]| + 1e-6 of the exactly rounded value when
 * scale * sum_d |q[d] K_t[d]| <= 60 for every token.
 *
 * Because seq_lens and block_table live on the device they cannot be
 * checked before the launch.  The kernels never read outside the arrays
 * described above: a sequence whose length is negative, above max_seq_len or
 * above max_pages_per_seq * page_size, or whose used block-table entries
 * name a page outside [0, num_pages), gets NaN in every output element;
 * other sequences are unaffected.
 */
#ifndef WQ_ATTENTION_H
#define WQ_ATTENTION_H

#include <stddef.h>
#include <stdint.h>

#include "wq.h"

#ifdef __cplusplus
extern "C" {
#endif

#define WQ_ATTN_HEAD_DIM 128                 /* the only head_dim supported */
#define WQ_ATTN_MAX_GROUP 8                  /* num_q_heads / num_kv_heads */
#define WQ_ATTN_MAX_KV_HEADS 256
#define WQ_ATTN_MAX_PAGE_SIZE 1024           /* a power of two */
#define WQ_ATTN_MAX_SEQ_LEN ((int64_t)1 << 22)
#define WQ_ATTN_MAX_SEQS ((int64_t)1 << 20)

/*
 * wq_paged_attention_workspace_size -- bytes of device workspace that
 * wq_paged_attention needs for these sizes (0 when none: the sequence is
 * then not split across workgroups).  Pure host function.
 * Errors: INVALID_ARG (null `bytes`, sizes out of range), UNSUPPORTED.
 */
wq_status wq_paged_attention_workspace_size(int64_t num_seqs, int64_t num_q_heads,
                                            int64_t num_kv_heads, int64_t head_dim,
                                            int64_t max_seq_len, size_t* bytes);

/*
 * wq_paged_attention -- out = attention of q over the paged cache.
 *
 *   q, out            16-byte aligned; out written, everything else read only.
 *   k_cache, v_cache  16-byte aligned.
 *   block_table, seq_lens  4-byte aligned.
 *   num_seqs          1 .. WQ_ATTN_MAX_SEQS.
 *   num_q_heads       a multiple of num_kv_heads, at most WQ_ATTN_MAX_GROUP
 *                     times it.
 *   num_kv_heads      1 .. WQ_ATTN_MAX_KV_HEADS.
 *   head_dim          WQ_ATTN_HEAD_DIM.
 *   page_size         a power of two, 1 .. WQ_ATTN_MAX_PAGE_SIZE.
 *   num_pages         1 .. 2^31 - 1 pages in each cache array.
 *   max_pages_per_seq row length of block_table, >= 1.
 *   max_seq_len       an upper bound of every L_s, 0 .. WQ_ATTN_MAX_SEQ_LEN and
 *                     at most max_pages_per_seq * page_size; it sizes the
 *                     launch, so a tight bound is faster.
 *   scale             finite; usually 1 / sqrt(head_dim).
 *   workspace         device memory of at least the size that
 *                     wq_paged_attention_workspace_size reports, 16-byte
 *                     aligned, owned by the caller, used only while the work
 *                     queued by this call runs (calls on one stream may share
 *                     it); may be NULL when that size is 0.
 * out must not overlap any input or the workspace.
 * Errors: INVALID_ARG, UNSUPPORTED (head_dim, group or page size),
 *         MISALIGNED, HIP.
 */
wq_status wq_paged_attention(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                             const int32_t* block_table, const int32_t* seq_lens, uint16_t* out,
                             int64_t num_seqs, int64_t num_q_heads, int64_t num_kv_heads,
                             int64_t head_dim, int64_t page_size, int64_t num_pages,
                             int64_t max_pages_per_seq, int64_t max_seq_len, float scale,
                             void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* WQ_ATTENTION_H */
