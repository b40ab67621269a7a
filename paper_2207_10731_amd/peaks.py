"""Measured bandwidth denominators of the roofline, per memory level.

The vendor publishes one figure for MI355X memory: 8 TB/s of HBM3E.  The
L2 (4 MiB per XCD) and the memory-side cache that sits in front of HBM have
no published peak, so the roofline at those levels uses rates measured here
with the kernels of libpss_bench.so (timed with events on the current
stream):

  read    streaming 16-byte loads by 8 workgroups per compute unit
  gather  random 64-byte reads (16 consecutive floats at a random 4-byte
          offset: the access of a chunk of Z = 16 weights)

from three buffers: one 2 MiB slice per XCD (each XCD re-reads its own slice,
which its L2 holds), a 128 MiB buffer (larger than the aggregate L2, held by
the memory-side cache after a first pass) and a 4 GiB buffer (HBM).
"""
from __future__ import annotations

import ctypes

import torch

from . import pss

L2_SLICE = 2 << 20     # bytes per XCD slice
CACHE_BUF = 128 << 20  # within the memory-side cache, beyond the aggregate L2
HBM_BUF = 4 << 30


def _time(fn, reps):
    fn()  # first pass brings the buffer to its level
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e-3 / reps


def measure(device=None) -> dict:
    """GB/s of streaming reads and of random 64-byte gathers at each level."""
    lib = pss.load_bench_library()
    dev = device or torch.device("cuda", torch.cuda.current_device())
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    sink = torch.zeros(256, dtype=torch.float32, device=dev)
    out = {}
    for level, nbytes, slices, passes, iters in (("l2", 8 * L2_SLICE, 1, 64, 512),
                                                  ("cache", CACHE_BUF, 0, 8, 512),
                                                  ("hbm", HBM_BUF, 0, 1, 256)):
        buf = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
        ptr = ctypes.c_void_p(buf.data_ptr())

        def rd():
            st = lib.pss_bench_read(ptr, nbytes, passes, slices, ctypes.c_void_p(sink.data_ptr()), s)
            if st != 0:
                raise RuntimeError(f"pss_bench_read failed: {st}")

        n = ctypes.c_int64(0)

        def ga():
            st = lib.pss_bench_gather(ptr, nbytes, iters, slices, 12345,
                                      ctypes.c_void_p(sink.data_ptr()), ctypes.byref(n), s)
            if st != 0:
                raise RuntimeError(f"pss_bench_gather failed: {st}")

        t_read = _time(rd, 3)
        t_gather = _time(ga, 3)
        out[f"{level}_read_gbs"] = nbytes * passes / t_read / 1e9
        out[f"{level}_gather_gbs"] = n.value * 64 / t_gather / 1e9
        del buf
    torch.cuda.empty_cache()
    return out


if __name__ == "__main__":
    for k, v in measure().items():
        print(f"{k}: {v:.0f} GB/s")
