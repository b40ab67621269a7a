/*
 * pss_bench.h - measurement helpers that sit beside the PSS layer, in a
 * library of their own (libpss_bench.so); none of them is part of the layer.
 *
 * pss_bench_copy is a plain streaming copy of known size, used to calibrate
 * hardware traffic counters (bytes fetched / written per dispatch) against
 * the bytes a kernel is known to move.  pss_bench_read and pss_bench_gather
 * measure the bandwidth denominators of the roofline at the memory level a
 * shared array lives in: a buffer split into one slice per XCD small enough
 * for that XCD's L2, a buffer larger than the chip's aggregate L2 but within
 * its memory-side cache, or one larger than both (HBM).  The caller times
 * them (events on `stream`) and divides the bytes moved by the time.
 * Every pointer is device memory owned by the caller; nothing is kept.
 */
#ifndef PSS_BENCH_H
#define PSS_BENCH_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* dst[0 .. bytes) = src[0 .. bytes) on `stream`; both device pointers,
 * 16-byte aligned, bytes a multiple of 16, non-overlapping.  Returns 0 on
 * success, 1 on bad arguments, 3 on a launch failure. */
int pss_bench_copy(void* dst, const void* src, size_t bytes, hipStream_t stream);

/* Streaming read of buf[0 .. bytes), `passes` times, by 8 resident
 * workgroups per compute unit with ordinary (cached) 16-byte loads.  With
 * xcd_slices != 0 the buffer is cut into 8 equal slices and the workgroups
 * of XCD x (workgroup b runs on XCD b mod 8) read only slice x, so a slice no
 * larger than one XCD's L2 is served by that L2 after the first pass.  Bytes
 * moved: bytes * passes.  buf 16-byte aligned; bytes a multiple of 16 (of
 * 128 with slices).  sink: device float[256], written only by a value the
 * caller's fill never produces.  Returns 0, 1 (bad arguments) or 3 (launch
 * failure). */
int pss_bench_read(const void* buf, size_t bytes, int passes, int xcd_slices, float* sink,
                   hipStream_t stream);

/* Random 64-byte gathers: every group of 16 lanes reads 16 consecutive
 * floats at `iters` pseudo-random 4-byte-aligned positions of its slice (the
 * access of a chunk of Z = 16 weights at a hashed base), slices as for
 * pss_bench_read.  *gathers (host) receives the number of 64-byte gathers
 * launched.  buf 4-byte aligned; bytes a multiple of 4 (of 32 with slices),
 * each slice between 32 and 2^32 floats.  Returns 0, 1 or 3. */
int pss_bench_gather(const void* buf, size_t bytes, int iters, int xcd_slices, uint32_t seed,
                     float* sink, int64_t* gathers, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* PSS_BENCH_H */
