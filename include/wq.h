/*
 * wq.h -- C ABI of the MI355X (gfx950) 4-bit group-quantized decode-linear
 * library.
 *
 * The operation is the decode-step linear layer of a 4-bit weight-quantized
 * decoder LLM (WebLLM, Sec. 1 and Sec. 3 / Table 1: token-by-token decoding
 * of 4-bit quantized 1-8B models; Sec. 2.3: weights converted ahead of time,
 * graph-level kernel fusion and operator-level GEMM tiling).  Dequantizing
 * the codes in registers inside the matrix-vector kernel is this library's
 * design, not a detail the paper gives:
 *
 *     y[m][n] = sum_k x[m][k] * w_hat[n][k],   w_hat[n][k] = s16[n][k/32] * (q[n][k] - 8)
 *
 * Weight format (this library's reading of "4-bit quantized"):
 *   - W is [N][K] (output features x input features), row-major.
 *   - K is split into groups of 32 consecutive elements of a row.
 *   - scale: s16 = fp16_rne(fp32(max|w over group| / 7)), stored as IEEE
 *     binary16 bit patterns, [N][K/32] row-major.
 *   - code: q = clamp(round_half_even(fp32(w / fp32(s16))) + 8, 0, 15);
 *     q = 8 for every element when s16 == 0.
 *   - packing: 8 codes per uint32, little-endian nibbles: element 8j+i of a
 *     row is bits [4i, 4i+4) of word j; packed_w is [N][K/8] row-major.
 * Activations x [M][K] and outputs y [M][N] are row-major IEEE binary16
 * passed as uint16_t bit patterns.
 *
 * Conventions shared by every entry point:
 *   - All data pointers are DEVICE pointers, allocated and owned by the
 *     caller; they must stay valid until the queued work has run (and, for
 *     work captured into a graph, for as long as the graph is replayed).
 *     The buffers the library owns itself are listed at wq_decode_linears.
 *   - `stream` is a hipStream_t passed as void*; NULL is the null stream.
 *     Calls are asynchronous and stream-ordered: they return after queuing
 *     work.  A device fault surfaces at the caller's next synchronization.
 *   - Every argument is validated on the host BEFORE any HIP call, so an
 *     invalid call returns an error without touching the device.
 *   - Return values are wq_status codes; wq_last_error_message() gives a
 *     human-readable description of the last failure on the calling thread.
 *   - Non-finite weights or activations give unspecified (but memory-safe)
 *     results.
 */
#ifndef WQ_H
#define WQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum wq_status {
    WQ_OK = 0,
    WQ_ERR_INVALID_ARG = 1,  /* null pointer, size <= 0 or too large, aliasing */
    WQ_ERR_UNSUPPORTED = 2,  /* group != 32, K % 32 != 0 */
    WQ_ERR_MISALIGNED = 3,   /* a pointer below its required alignment */
    WQ_ERR_HIP = 4           /* the HIP runtime reported an error */
} wq_status;

/* Largest accepted sizes. */
#define WQ_MAX_N ((int64_t)0x7fffffff)
#define WQ_MAX_K ((int64_t)0x7fffffe0)
#define WQ_MAX_M ((int64_t)65535)
#define WQ_MAX_LINEARS ((int64_t)65536)

/* Static string naming a status code ("WQ_OK", ...); "WQ_UNKNOWN_STATUS" for
 * values outside the enum.  Never NULL. */
const char* wq_status_string(int status);

/* Description of the last non-OK status returned on the calling thread
 * (thread-local, overwritten by the next failing call).  Never NULL. */
const char* wq_last_error_message(void);

/* Library ABI version: 100 * major + minor. */
int wq_version(void);

/*
 * wq_pack -- quantize fp32 weights to the 4-bit format above (the ahead-of-
 * time weight conversion of Sec. 2.3; 4-bit models of Table 1).
 *
 *   w         [N][K] fp32, device, 16-byte aligned, read only.
 *   packed_w  [N][K/8] uint32, device, 16-byte aligned, written.
 *   scales    [N][K/32] fp16 bits, device, 2-byte aligned, written.
 *   N, K      1 <= N <= WQ_MAX_N, 32 <= K <= WQ_MAX_K.
 *   group     must be 32.
 * Output is bit-exact: IEEE division, round-half-even, fp16 subnormals kept.
 * Errors: INVALID_ARG (null, N or K <= 0 or too large, output overlapping w),
 *         UNSUPPORTED (group != 32, K % 32 != 0), MISALIGNED, HIP.
 */
wq_status wq_pack(const float* w, uint32_t* packed_w, uint16_t* scales,
                  int64_t N, int64_t K, int64_t group, void* stream);

/*
 * wq_gemv -- y = x * dequant(W)^T for a small batch of activations (the
 * decode-step linear, Sec. 1 / Table 1; dequantization fused in registers).
 *
 *   packed_w  [N][K/8] uint32, device, 16-byte aligned, read only.
 *   scales    [N][K/32] fp16 bits, device, 2-byte aligned, read only.
 *   x         [M][K] fp16 bits, device, 16-byte aligned, read only.
 *   y         [M][N] fp16 bits, device, 2-byte aligned, written.
 *   N, K, M   1 <= N <= WQ_MAX_N, 32 <= K <= WQ_MAX_K, 1 <= M <= WQ_MAX_M.
 *   group     must be 32.
 * Accumulation is fp32; each output is rounded once to fp16 (round to
 * nearest even).  For M <= 2 every product is exact.  For M >= 3 (matrix
 * cores) each scaled weight (q - 8) * s is first rounded to fp16 (relative
 * error <= 2^-11); this needs |(q - 8) * s| <= 65504, i.e. scales below 8188,
 * and larger scales give infinities on that path.  Per element the result is
 * within 1e-3 * sum_k |w_hat[n][k] x[m][k]| + 1e-5 of the exactly rounded
 * value.
 * y must not overlap x, packed_w or scales.
 * Errors: INVALID_ARG, UNSUPPORTED, MISALIGNED, HIP (as for wq_pack).
 */
wq_status wq_gemv(const uint32_t* packed_w, const uint16_t* scales,
                  const uint16_t* x, uint16_t* y,
                  int64_t N, int64_t K, int64_t M, int64_t group, void* stream);

/* One linear layer of a decode step; pointers and sizes as for wq_gemv. */
typedef struct wq_linear {
    const uint32_t* packed_w;
    const uint16_t* scales;
    const uint16_t* x;
    uint16_t* y;
    int64_t N;
    int64_t K;
} wq_linear;

/*
 * wq_decode_linears -- run linears[0 .. count) in order on one stream: one
 * decode step's linear layers (the per-token work whose throughput Table 1
 * reports).  Linear i may read, as its x, the y written by any linear j < i,
 * and may overwrite any earlier linear's x or y: the result is that of
 * running the linears one after another.  No y may overlap the x of the
 * same linear, nor the packed_w or scales of any linear in the list.
 *
 *   linears   HOST array of `count` descriptors; read during the call
 *             only, so it may be freed or reused as soon as the call returns.
 *   count     1 <= count <= WQ_MAX_LINEARS.
 *   M, group  shared by all linears (1 <= M <= WQ_MAX_M, group == 32).
 *
 * Library-owned resources.  For M <= 64 the call turns the list into a
 * launch plan (about 76 bytes per linear) that the kernels read from device
 * memory.  Per (device, stream) pair it is called with, the library keeps,
 * until the process ends: up to 32 device plan buffers holding the plans of
 * the most recently used distinct descriptor lists, any number of frozen
 * plan buffers (below), two pinned host staging buffers, and two events.
 * They are allocated on first use and grown when a longer list needs it.
 * A list whose plan is already resident is launched without any copy.
 *
 * Host blocking.  The call returns after queuing work, except that it waits
 * (a) for the stream to drain when a plan buffer must grow, and (b) for the
 * older of two uploads still in flight when a third distinct list arrives
 * before the device has read either.  Two lists used alternately never wait.
 *
 * Stream capture.  When `stream` is capturing, the call records kernel
 * launches only: if the list's plan is resident (the same call was made on
 * this stream outside capture before), its buffer is frozen -- never
 * rewritten or freed -- so the captured graph stays valid for the life of the
 * process, whatever calls follow.  Otherwise the call returns
 * WQ_ERR_UNSUPPORTED and captures nothing; wq_decode_linears_noalloc needs
 * no prior call.
 *
 * Errors: as wq_gemv, checked for every descriptor before anything runs;
 * UNSUPPORTED as above.
 */
wq_status wq_decode_linears(const wq_linear* linears, int64_t count,
                            int64_t M, int64_t group, void* stream);

/* Limits of wq_decode_linears_noalloc. */
#define WQ_NOALLOC_MAX_LINEARS ((int64_t)1024)
#define WQ_NOALLOC_SCRATCH_BYTES ((int64_t)131072)

/*
 * wq_decode_linears_noalloc -- wq_decode_linears for callers that cannot
 * allocate: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Same arguments, kernels and results (bit for bit) as
 * wq_decode_linears; it calls no hipMalloc, hipFree or other allocating
 * routine and takes no host or device memory of its own beyond fixed static
 * storage.
 *
 * The launch plan lives in a fixed device array of WQ_NOALLOC_SCRATCH_BYTES
 * per device, held until the process ends (its address is looked up on the
 * first call made with that device current).  Each call rewrites the array
 * with its own plan through small kernels, queued on `stream` ahead of the
 * GEMV launches, whose launch arguments carry the plan bytes: no host memory
 * is read after the call returns, so a call captured into a graph carries its
 * plan and replays correctly after any other calls.  All calls on one device
 * share the array: calls or graph replays that overlap in time on different
 * streams of one device race and give undefined results.  Calls on one
 * stream are ordered and safe.  The host waits for nothing.
 *
 * Errors: as wq_decode_linears; INVALID_ARG also when count exceeds
 * WQ_NOALLOC_MAX_LINEARS (the plan of that many linears, at most 128 bytes
 * per linear, always fits the array); UNSUPPORTED on a device numbered 64 or
 * above.
 */
wq_status wq_decode_linears_noalloc(const wq_linear* linears, int64_t count,
                                    int64_t M, int64_t group, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* WQ_H */
