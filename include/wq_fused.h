/*
 * wq_fused.h -- C ABI of a decode step's 4-bit linears with the elementwise
 * work around them fused in, in the same library as wq.h (libwq.so; status
 * codes and error messages are shared with it).
 *
 * The paper's compiler fuses kernels at the graph level (Sec. 2.3).  In the
 * Llama-class decoders of Table 1 the work next to each decode linear is an
 * RMS normalisation of its input (QKV, gate/up and the final projection), the
 * SiLU-gated product of the gate/up output (the down projection's input), a
 * residual addition of its output (O and down) and the choice of the next
 * token from the logits.  Here each linear may take a prologue, applied to x
 * while x is staged, and a residual, added to the fp32 result before the one
 * fp16 rounding of y:
 *
 *   WQ_PROLOGUE_NONE      x_eff[k] = x[k]                          x has K entries
 *   WQ_PROLOGUE_RMSNORM   x_eff[k] = fp16(x[k] / sqrt(mean_j x[j]^2 + eps)
 *                                         * norm_weight[k])         x has K entries
 *   WQ_PROLOGUE_SILU_MUL  x_eff[k] = fp16(silu(x[k]) * x[K + k]),
 *                         silu(a) = a / (1 + exp(-a))               x has 2K entries
 *
 *   y[n] = fp16(sum_k w_hat[n][k] * x_eff[k] + residual[n])   (residual optional)
 *
 * The weight format and w_hat are those of wq.h.  Batch 1 (one token).  The
 * prologue's reductions and products are fp32, as is the dot product; x_eff
 * is rounded to fp16 as the linear's input.  Per element y is within
 * 2e-3 * (sum_k |w_hat[n][k] x_eff[k]| + |residual[n]|) + 1e-5 of the exactly
 * rounded value.
 */
#ifndef WQ_FUSED_H
#define WQ_FUSED_H

#include <stdint.h>

#include "wq.h"

#ifdef __cplusplus
extern "C" {
#endif

#define WQ_PROLOGUE_NONE 0
#define WQ_PROLOGUE_RMSNORM 1
#define WQ_PROLOGUE_SILU_MUL 2

/* Largest K of a fused linear: 512 groups of 32. */
#define WQ_FUSED_MAX_K ((int64_t)16384)

/* One linear of a fused chain.  All pointers are DEVICE pointers owned by the
 * caller. */
typedef struct wq_fused_linear {
    const uint32_t* packed_w;     /* [N][K/8], 16-byte aligned */
    const uint16_t* scales;       /* [N][K/32] fp16 bits, 2-byte aligned */
    const uint16_t* x;            /* [K] ([2K] for SILU_MUL) fp16 bits, 16-byte aligned */
    uint16_t* y;                  /* [N] fp16 bits, 2-byte aligned, written */
    const uint16_t* norm_weight;  /* [K] fp16 bits, 16-byte aligned (RMSNORM only; else ignored) */
    const uint16_t* residual;     /* [N] fp16 bits, 2-byte aligned, or NULL; may be y itself */
    int64_t N;                    /* 1 .. WQ_MAX_N */
    int64_t K;                    /* a multiple of 32, 32 .. WQ_FUSED_MAX_K */
    int32_t prologue;             /* WQ_PROLOGUE_* */
    float eps;                    /* RMSNORM: finite and >= 0 (and mean(x^2) + eps > 0) */
} wq_fused_linear;

/*
 * wq_fused_linears -- run linears[0 .. count) in order on one stream, each
 * a separate launch that starts after the previous one has finished: linear
 * i may read, as its x, norm weight or residual, anything an earlier linear
 * wrote.  This is a decode layer chain such as
 *   RMSNorm -> QKV,  (attention),  O + residual,  RMSNorm -> gate/up,
 *   SiLU-mul -> down + residual,  ...,  RMSNorm -> lm_head.
 *
 *   linears   HOST array of `count` descriptors, read during the call only.
 *   count     1 .. WQ_MAX_LINEARS.
 *   argmax    DEVICE int32 pointer, or NULL.  When given, after the last
 *             linear the index of the largest element of its y (the
 *             smallest such index on ties; NaN elements never win; -1 when
 *             all are NaN) is written there.
 *   group     must be 32.
 * A linear's y must not overlap its own x or norm weight, nor the packed_w or
 * scales of any linear; its residual is either exactly y or does not overlap
 * y; argmax must not overlap any array of the chain.
 * Errors: INVALID_ARG (null, sizes, prologue, eps, aliasing), UNSUPPORTED
 * (group, K % 32, K above WQ_FUSED_MAX_K, codes of one linear above 4 GiB),
 * MISALIGNED, HIP.  Every descriptor is checked before anything runs.
 */
wq_status wq_fused_linears(const wq_fused_linear* linears, int64_t count, int32_t* argmax,
                           int64_t group, void* stream);

/*
 * wq_fused_check -- synchronize `stream`, then report whether a persistent
 * chain (below) on the current device has given up since the last check.
 * Returns WQ_ERR_HIP in that case (and clears the condition), WQ_OK
 * otherwise, or WQ_ERR_HIP for a runtime error of the synchronization.
 *
 * How wq_fused_linears runs a chain.  By default each linear is one launch
 * (the per-linear path).  With WQ_FUSED_PERSISTENT=1 in the environment
 * (read at every call), when the current device supports cooperative
 * launches, the stream is not capturing, the chain has fewer than 32767
 * linears, every linear's rows are of one of the compiled shapes (up to 256
 * groups, K <= 8192, codes below 2 GiB, at most 512 rows per wave), every x
 * and residual is either an input from outside the chain or lies inside the
 * output of one earlier linear, and no norm weight is an output of the
 * chain, the chain is instead ONE cooperative launch of a persistent kernel
 * (one workgroup per CU) followed by a small copy kernel.  Inside it, outputs
 * pass between workgroups through a library buffer as tagged words, which
 * the consumers read until the tags show them complete, while the weights
 * of the next linears keep streaming; the caller's y buffers are written
 * only by the copy kernel at the end.  Results are bit-identical to the
 * per-linear path.  (It is not the default: on MI355X a boundary inside it
 * costs about 5 us, two agent-scope memory round trips, against about
 * 3 us for a kernel boundary of the per-linear path, so a whole 3B-class
 * token takes longer this way.)
 *
 * The persistent path's library memory is part of the resident plan of the
 * (device, stream) pair (see wq_decode_linears in wq.h): the plan, and 4
 * bytes per output element of the chain, zeroed when the plan is set up.
 * Two persistent chains must not run at the same time on one stream's plan.
 * Every wait in the kernel is bounded (half a second; the environment
 * variable WQ_CHAIN_TIMEOUT_TICKS sets it in clock ticks, for tests): when a
 * wait runs out, every later wait of the launch gives up at once, every wave
 * ends, that call's outputs are undefined, and the next wq_fused_check
 * reports it.
 */
wq_status wq_fused_check(void* stream);

#ifdef __cplusplus
}
#endif

#endif /* WQ_FUSED_H */
