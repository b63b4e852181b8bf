/*
 * wq_probe.h -- measurement probe in the same library as wq.h (libwq.so;
 * status codes and error messages shared with it).  It computes nothing of
 * the method: it gives the bandwidth a plain streaming read reaches on the
 * device, the practical ceiling the decode kernels' HBM figures are read
 * against.
 */
#ifndef WQ_PROBE_H
#define WQ_PROBE_H

#include <stdint.h>

#include "wq.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * wq_stream_read -- read `bytes` of device memory at `buf` once, in 16-byte
 * non-temporal loads: up to 1024 workgroups of 256 threads, each streaming
 * its own contiguous range (4 loads in flight per thread), the access
 * pattern of the decode kernels.  The loaded data is folded into one word
 * per workgroup that is stored to
 * sink[blockIdx] only in the (practically impossible) case that it equals
 * 0x9E3779B9, so that no load can be optimised away and almost nothing is
 * written.
 *
 *   buf    DEVICE pointer, 16-byte aligned, `bytes` readable bytes.
 *   bytes  a positive multiple of 16.
 *   sink   DEVICE pointer to 1024 uint32 (the largest grid), 4-byte aligned.
 * Asynchronous on `stream` like every call of the library.
 * Errors: INVALID_ARG (null, bytes <= 0 or not a multiple of 16),
 *         MISALIGNED, HIP.
 */
wq_status wq_stream_read(const void* buf, int64_t bytes, uint32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* WQ_PROBE_H */
