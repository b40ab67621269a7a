"""Shape sweeps of the PSS layer on one GPU (the paper's micro-benchmark setup).

The paper times a single embedding table looked up with batch 10240 and
d = 128, with the loss taken as the sum of all retrieved elements (so the
output gradient is all ones), while varying the chunk size Z and the
compression (original table size n*d over |M|); it reports that larger
chunks help, and that dense gradients win at high compression while sparse
gradients cost the same at every compression (Sec. 3, appendix
observations).  This module measures the same sweeps here:

  python -m paper_2207_10731_amd.sweep chunk      forward/backward vs Z
  python -m paper_2207_10731_amd.sweep crossover  dense vs sparse backward vs |M|
  python -m paper_2207_10731_amd.sweep compress   post-hoc M = S E of a given
                                                  table (Sec. 2.4): time per
                                                  backward variant and the
                                                  empirical eps of Def. 2
  python -m paper_2207_10731_amd.sweep address    SORTED backward grouped by
                                                  token vs deposited by
                                                  address, vs Z and |M|, on a
                                                  26-table one-hot batch of
                                                  uniform indices

Inputs: n = 10^7 rows, one uniform index per sample, grad_out = 1.
Each point: median of `--reps` timed calls (HIP events on the stream the
library launches on) after warm-up.  Output: one markdown table on stdout.
"""
from __future__ import annotations

import argparse
import os
import sys

import numpy as np
import torch

from . import pss

ROWS = 10_000_000
BATCH = 10240
DIM = 128


def _time(fn, reps, warmup=3):
    for _ in range(warmup):
        fn()
    ts = []
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) * 1e3)
    return float(np.median(ts))


class Point:
    def __init__(self, M, Z, seed=7, optimizer="sgd", dev="cuda"):
        rng = np.random.default_rng(seed)
        self.M, self.Z = int(M), int(Z)
        self.idx = torch.from_numpy(rng.integers(0, ROWS, BATCH, dtype=np.int64)).to(dev)
        self.off = torch.arange(BATCH + 1, dtype=torch.int64, device=dev)
        self.w = torch.from_numpy(rng.uniform(-0.01, 0.01, self.M).astype(np.float32)).to(dev)
        self.state = torch.zeros(self.M, device=dev) if optimizer == "adagrad" else None
        self.grad = torch.ones((BATCH, DIM), device=dev)
        self.out = torch.empty((BATCH, DIM), device=dev)
        self.seed = seed

    def hp(self, flags):
        return pss.make_hash_params(self.seed, num_tables=1, batch=BATCH, num_indices=BATCH,
                                    flags=flags)

    def forward(self):
        pss.pss_forward(self.w, self.M, self.Z, DIM, self.hp(pss.PSS_BWD_AUTO), self.idx, self.off,
                        self.out)

    def backward(self, flags, lr=1e-4):
        pss.pss_backward_update(self.w, self.state, self.M, self.Z, DIM, self.hp(flags), self.idx,
                                self.off, self.grad, lr)


def chunk_sweep(reps):
    print("| Z | compression | M | forward us | backward (sorted) us | backward (sparse) us |")
    print("|---|---|---|---|---|---|")
    for comp in (1000, 10000):
        M = ROWS * DIM // comp
        for Z in (1, 2, 4, 8, 16, 32, 64, 128):
            pt = Point(M, Z)
            f = _time(pt.forward, reps)
            b = _time(lambda: pt.backward(pss.PSS_BWD_SORTED), reps)
            s = _time(lambda: pt.backward(pss.PSS_BWD_SPARSE), reps)
            print(f"| {Z} | {comp}x | {M} | {f:.1f} | {b:.1f} | {s:.1f} |", flush=True)


def crossover_sweep(reps):
    print("| compression | M | optimizer | dense (sorted) us | dense (atomic) us | sparse us |")
    print("|---|---|---|---|---|---|")
    for opt in ("adagrad", "sgd"):
        for comp in (10, 100, 1000, 10000, 100000):
            M = ROWS * DIM // comp
            pt = Point(M, 32, optimizer=opt)
            d = _time(lambda: pt.backward(pss.PSS_BWD_SORTED), reps)
            a = _time(lambda: pt.backward(pss.PSS_BWD_ATOMIC), reps)
            s = _time(lambda: pt.backward(pss.PSS_BWD_SPARSE), reps)
            print(f"| {comp}x | {M} | {opt} | {d:.1f} | {a:.1f} | {s:.1f} |", flush=True)


def compress_sweep(reps, Z=32):
    """One table of ROWS x DIM entries drawn i.i.d. N(0, 1).  For each
    compression: time of compress_table per backward variant (and the rate
    at which table entries are read), then the per-row eps of Def. 2,
    ||(S e_i)^T M - E_i||, against its expectation over the draw of E,
    sqrt(sum_m load(m)(load(m) - 1) / n) with load from compressing ones."""
    g = torch.Generator(device="cuda").manual_seed(11)
    E = torch.randn((1, ROWS, DIM), device="cuda", generator=g)
    ones = torch.ones_like(E)
    norm = E[0].norm(dim=1).mean().item()
    print(f"<!-- Z = {Z}; mean ||E_i|| = {norm:.3f} -->")
    print("| compression | M | sparse us | sorted us | atomic us | entries/s (best) "
          "| mean eps | p99 eps | max eps | sqrt E[eps^2] | mean eps / mean norm |")
    print("|---|---|---|---|---|---|---|---|---|---|---|")
    for comp in (10, 100, 1000, 10000):
        M = ROWS * DIM // comp
        hp = pss.make_hash_params(21, num_tables=1, batch=ROWS, num_indices=ROWS)
        out = torch.empty(M, device="cuda")
        t = {}
        for name, v in (("sparse", pss.PSS_BWD_SPARSE), ("sorted", pss.PSS_BWD_SORTED),
                        ("atomic", pss.PSS_BWD_ATOMIC)):
            t[name] = _time(lambda: pss.compress_table(E, M, Z, hp, variant=v, out=out), reps, 1)
        pss.compress_table(E, M, Z, hp, out=out)
        R = pss.lookup_rows(out, M, Z, DIM, 1, ROWS, hp)
        eps = (R - E).norm(dim=2).flatten()
        del R
        load = pss.compress_table(ones, M, Z, hp, variant=pss.PSS_BWD_SORTED)
        expect = ((load.double() * (load.double() - 1)).sum() / ROWS).sqrt().item()
        del load
        e_sorted = eps.sort().values
        best = min(t.values())
        print(f"| {comp}x | {M} | {t['sparse']:.0f} | {t['sorted']:.0f} | {t['atomic']:.0f} "
              f"| {ROWS * DIM / best * 1e6:.3g} | {eps.mean().item():.3f} "
              f"| {e_sorted[int(0.99 * ROWS)].item():.3f} | {e_sorted[-1].item():.3f} "
              f"| {expect:.3f} | {eps.mean().item() / norm:.3f} |", flush=True)
        del eps, e_sorted, out


def address_sweep(reps, tables=26, batch=65536, rows=40_000_000):
    """Backward (SGD on float32, N(0, 1) output gradient) of a one-hot batch
    of `tables` tables x `batch` samples with uniform indices over `rows`
    rows: the SORTED variant grouped by token against the same with
    PSS_DEPOSIT_BY_ADDRESS, for chunk sizes 1..16 and two array sizes."""
    rng = np.random.default_rng(5)
    n = tables * batch
    idx = torch.from_numpy(rng.integers(0, rows, n, dtype=np.int64)).cuda()
    off = torch.arange(n + 1, dtype=torch.int64, device="cuda")
    g = torch.Generator(device="cuda").manual_seed(6)
    grad = torch.randn((batch, tables * DIM), device="cuda", generator=g)
    print("| M | Z | by token us | by address us |")
    print("|---|---|---|---|")
    for M in (2_500_000, 1_000_000_000):
        w = torch.zeros(M, device="cuda")
        for Z in (1, 2, 4, 8, 16):
            t = {}
            for name, fl in (("token", pss.PSS_BWD_SORTED),
                             ("address", pss.PSS_BWD_SORTED | pss.PSS_DEPOSIT_BY_ADDRESS)):
                hp = pss.make_hash_params(9, num_tables=tables, batch=batch, num_indices=n,
                                          flags=fl)
                t[name] = _time(lambda: pss.pss_backward_update(w, None, M, Z, DIM, hp, idx, off,
                                                                grad, 0.1), reps, 2)
            print(f"| {M} | {Z} | {t['token']:.0f} | {t['address']:.0f} |", flush=True)
        del w


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("mode", choices=["chunk", "crossover", "compress", "address"])
    ap.add_argument("--reps", type=int, default=20)
    a = ap.parse_args(argv)
    assert torch.cuda.is_available(), "the sweep needs a GPU"
    if a.mode == "address":
        print(f"<!-- {torch.cuda.get_device_name(0)}; 26 tables x 65536 samples, one uniform "
              f"index in [0, 4e7) each, d = {DIM}, grad_out N(0, 1), SGD, median of {a.reps} -->")
    else:
        print(f"<!-- {torch.cuda.get_device_name(0)}; n = {ROWS} rows, batch {BATCH}, d = {DIM}, "
              f"grad_out = 1, median of {a.reps} -->")
    {"chunk": chunk_sweep, "crossover": crossover_sweep, "compress": compress_sweep,
     "address": address_sweep}[a.mode](a.reps)


if __name__ == "__main__":
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    main()
