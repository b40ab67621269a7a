"""Runs pss_bench_copy on a buffer of known size (default 1 GiB), a few times.

Profile it beside a workload to turn the FETCH_SIZE / WRITE_SIZE counters
(KiB per dispatch) into bytes: the copy moves exactly `--mib` MiB each way.
Usage: python -m paper_2207_10731_amd.calib_copy [--mib 1024] [--reps 3]
"""
import argparse
import ctypes
import sys

import torch

from . import pss


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--mib", type=int, default=1024)
    ap.add_argument("--reps", type=int, default=3)
    a = ap.parse_args()
    lib = pss.load_bench_library()
    nbytes = a.mib << 20
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    for _ in range(a.reps):
        st = lib.pss_bench_copy(ctypes.c_void_p(dst.data_ptr()), ctypes.c_void_p(src.data_ptr()), nbytes, s)
        if st != 0:
            sys.exit(f"pss_bench_copy failed: {st}")
    torch.cuda.synchronize()
    assert torch.equal(dst[:1024], src[:1024])
    print(f"copied {a.mib} MiB x {a.reps}")


if __name__ == "__main__":
    main()
