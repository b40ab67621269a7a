/*
 * pss_bench.h - measurement helpers that sit beside the PSS layer.
 *
 * pss_bench_copy is a plain streaming copy of known size, used to calibrate
 * hardware traffic counters (bytes fetched / written per dispatch) against
 * the bytes a kernel is known to move.  It is not part of the layer.
 */
#ifndef PSS_BENCH_H
#define PSS_BENCH_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* dst[0 .. bytes) = src[0 .. bytes) on `stream`; both device pointers,
 * 16-byte aligned, bytes a multiple of 16, non-overlapping.  Returns 0 on
 * success, 1 on bad arguments, 3 on a launch failure. */
int pss_bench_copy(void* dst, const void* src, size_t bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* PSS_BENCH_H */
