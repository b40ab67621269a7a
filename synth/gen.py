"""Seeded generators: cardinalities, bag lengths, indices, weights, gradients.

Every stream is drawn from ``numpy.random.default_rng([data_seed, stream,
batch])`` so that each component is reproducible on its own, whatever sizes
the others were drawn with.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .configs import Workload

_CARD, _LEN, _IDX, _W, _GRAD = 0, 1, 2, 3, 4


def _rng(wl: Workload, stream: int, batch: int = 0) -> np.random.Generator:
    return np.random.default_rng([wl.data_seed, stream, batch])


def cardinalities(wl: Workload) -> np.ndarray:
    """Rows per table (int64 [T])."""
    kind, *args = wl.cardinality.split(":")
    if kind == "fixed":
        return np.full(wl.T, int(args[0]), dtype=np.int64)
    if kind == "loguniform":
        lo, hi = float(args[0]), float(args[1])
        u = _rng(wl, _CARD).uniform(np.log(lo), np.log(hi), wl.T)
        return np.clip(np.rint(np.exp(u)), lo, hi).astype(np.int64)
    raise ValueError(wl.cardinality)


def bag_lengths(wl: Workload, B: int, batch: int = 0) -> np.ndarray:
    """Items per bag, table-major (bag g = t*B + b): int64 [T*B]."""
    if wl.bag == "one":
        return np.ones(wl.T * B, dtype=np.int64)
    kind, mean, lo, hi = wl.bag.split(":")
    assert kind == "poisson"
    lens = _rng(wl, _LEN, batch).poisson(float(mean), wl.T * B)
    return np.clip(lens, int(lo), int(hi)).astype(np.int64)


def _zipf_truncated(rng: np.random.Generator, s: float, n: int, size: int) -> np.ndarray:
    """Zipf(s) ranks restricted to 1..n by rejection; returned as rows rank-1."""
    out = rng.zipf(s, size)
    bad = out > n
    while bad.any():
        out[bad] = rng.zipf(s, int(bad.sum()))
        bad = out > n
    return (out - 1).astype(np.int64)


def indices_for(wl: Workload, lengths: np.ndarray, B: int, batch: int = 0) -> np.ndarray:
    """Token indices, table by table, following ``lengths`` (int64 [N])."""
    card = cardinalities(wl)
    rng = _rng(wl, _IDX, batch)
    per_table = lengths.reshape(wl.T, B).sum(axis=1)
    parts = []
    for t in range(wl.T):
        n = int(per_table[t])
        if wl.index_dist == "uniform":
            parts.append(rng.integers(0, card[t], n, dtype=np.int64))
        else:
            kind, s = wl.index_dist.split(":")
            assert kind == "zipf"
            parts.append(_zipf_truncated(rng, float(s), int(card[t]), n))
    return np.concatenate(parts) if parts else np.zeros(0, dtype=np.int64)


def make_weights(wl: Workload, M: int | None = None) -> np.ndarray:
    """Initial shared array, U(-0.01, 0.01).

    float32 [M] for f32 storage; for bf16 storage the float32 draw rounded to
    bfloat16 by torch (nearest-even), returned as uint16 bit patterns.
    """
    M = wl.M if M is None else M
    w = _rng(wl, _W).random(M, dtype=np.float32) * np.float32(0.02) - np.float32(0.01)
    if wl.weight_dtype == "f32":
        return w
    import torch
    return torch.from_numpy(w).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def make_grad(wl: Workload, B: int | None = None, batch: int = 0) -> np.ndarray:
    """Upstream gradient of the pooled output, N(0, 1) float32 [B, T*d]."""
    B = wl.B if B is None else B
    return _rng(wl, _GRAD, batch).standard_normal((B, wl.T * wl.d), dtype=np.float32)


@dataclass
class Inputs:
    indices: np.ndarray   # int64 [N]
    offsets: np.ndarray   # int64 [T*B + 1]
    B: int

    @property
    def N(self) -> int:
        return int(self.indices.shape[0])


def make_inputs(wl: Workload, B: int | None = None, batch: int = 0) -> Inputs:
    """One batch of bags: CSR offsets over table-major bags and their indices."""
    B = wl.B if B is None else B
    lens = bag_lengths(wl, B, batch)
    offsets = np.zeros(wl.T * B + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    idx = indices_for(wl, lens, B, batch)
    return Inputs(indices=idx, offsets=offsets, B=B)
