"""GPU parity of the run sums deposited by address (PSS_DEPOSIT_BY_ADDRESS
with chunks of 64 elements or more): the lookups are grouped by token, every run sum becomes one record
per chunk, the records are radix-sorted by address tile and each tile sums
its chunks in LDS and applies the optimizer in place (Alg. 1's dense branch,
the deposit of a token's summed gradient at its chunk's addresses).

Shapes put the array at exactly one tile (2^14 elements), one element past
it, a last tile shorter than a chunk (chunks of the tile before it cross
that whole tile and wrap to element 0), an array shorter than a tile and an
array exactly one chunk long (every chunk wraps within it), across 123
tiles with a ragged last one; whole-row chunks (Z = d = 128) and two chunks
per row (Z = 64); Zipf-skewed tokens whose runs span several 256-pair
pieces; bags of several items; every option; SGD on float32 and bfloat16
storage and Adagrad; the grouping made ahead by pss_prepare_backward; a
grad = 1 case whose result is an integer count, equal bit for bit; and the
same update run twice from the same state, equal bit for bit (every sum is
taken in a fixed order).
"""
import numpy as np
import pytest
import torch

import synth
from oracle import pss_oracle as o
from paper_2207_10731_amd import pss
import parity
from parity import Layer

pytestmark = pytest.mark.gpu

RUNS = pss.PSS_BWD_SORTED | pss.PSS_DEPOSIT_BY_ADDRESS
C5 = synth.get("c5")

# name: (workload, B, M, Z)
SHAPES = {
    "rowhash-2M": (C5, 300, 2_000_003, 128),
    "one-tile": (C5, 60, 16384, 128),
    "tile-plus-one": (C5, 60, 16385, 128),
    "short-last-tile": (C5, 60, 2 * 16384 + 50, 128),
    "small": (C5, 40, 1000, 128),
    "one-chunk": (C5, 20, 128, 128),
    "z64-two-chunks": (synth.get("c2"), 300, 2_500_000, 64),
    "multihot-z64": (synth.get("c3"), 30, 2_000_003, 64),
}


def _layer(shape, flags=RUNS, **kw):
    wl, B, M, Z = SHAPES[shape]
    wl = wl.scaled(M=M, Z=Z, **kw.pop("wl", {}))
    print(f"runs case {shape}: B={B} M={M} Z={Z} {kw}", flush=True)
    return Layer(wl, B=B, flags=flags, **kw)


def _check(L, lr=None):
    grad = synth.make_grad(L.wl, L.B, batch=0)
    L.backward(grad, lr=lr)
    w_ref, s_ref, G, A, _ = L.ref_backward(grad, lr=lr)
    s_gpu = None if L.state is None else L.state.cpu().numpy()
    parity.check_update(L, L.weights(), s_gpu, w_ref, s_ref, G, A, L.wl.lr if lr is None else lr)


@pytest.mark.parametrize("shape", list(SHAPES))
def test_runs_update(shape):
    """The workload's own optimizer and storage (bfloat16 + Adagrad on the
    row-hash shapes, float32 SGD on the one-hot one, Adagrad on the
    multi-hot one)."""
    _check(_layer(shape))


@pytest.mark.parametrize("shape", ["rowhash-2M", "short-last-tile", "z64-two-chunks"])
def test_runs_adagrad_f32(shape):
    _check(_layer(shape, wl=dict(optimizer="adagrad", weight_dtype="f32", lr=0.01), s0=0.1))


@pytest.mark.parametrize("shape", ["rowhash-2M", "one-chunk"])
def test_runs_sgd_bf16(shape):
    _check(_layer(shape, wl=dict(optimizer="sgd", weight_dtype="bf16", lr=0.1)))


OPTS = {
    "pm1": dict(sign="pm1"),
    "sparse": dict(sign="sparse"),
    "mean": dict(mean=True),
    "i32": dict(idx32=True),
    "bf16rows": dict(rows_bf16=True),
    "all": dict(sign="sparse", mean=True, idx32=True, rows_bf16=True),
}


@pytest.mark.parametrize("opt", list(OPTS))
@pytest.mark.parametrize("shape", ["z64-two-chunks", "multihot-z64"])
def test_runs_options(shape, opt):
    _check(_layer(shape, **OPTS[opt]))


@pytest.mark.parametrize("shape", ["rowhash-2M", "short-last-tile", "one-chunk", "multihot-z64"])
def test_runs_counts_bit_exact(shape):
    """w = 0, grad = 1, lr = 1, SGD on float32: every updated weight is minus
    the number of reads of that element, an integer the tile sums reach
    exactly in any order; untouched elements keep +0.0."""
    wl, B, M, Z = SHAPES[shape]
    wl = wl.scaled(M=M, Z=Z, optimizer="sgd", weight_dtype="f32")
    L = Layer(wl, B=B, flags=RUNS, w=np.zeros(M, dtype=np.float32))
    ones = np.ones((B, wl.T * wl.d), dtype=np.float32)
    L.backward(ones, lr=1.0)
    _, _, _, _, cnt = L.ref_backward(ones, lr=1.0)
    got = L.weights()
    assert np.array_equal(got, (-cnt).astype(np.float32))
    assert not np.signbit(got[cnt == 0]).any()


@pytest.mark.parametrize("shape", ["rowhash-2M", "multihot-z64"])
def test_runs_with_prepared_grouping(shape):
    """pss_prepare_backward, the forward, then the backward: the run sums
    are taken from the grouping made ahead."""
    L = _layer(shape)
    wl = L.wl
    g = synth.make_grad(wl, B=L.B)
    pss.pss_prepare_backward(wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets)
    L.forward()
    _check(L)


def test_runs_twice_in_a_row():
    """Two updates on one layer (the kept scratch is reused; the second
    call sees the first one's weights and state)."""
    L = _layer("rowhash-2M")
    wl = L.wl
    for batch in range(2):
        grad = synth.make_grad(wl, L.B, batch=batch)
        L.backward(grad)
        w_ref, s_ref, G, A, _ = L.ref_backward(grad)
        s_gpu = L.state.cpu().numpy()
        parity.check_update(L, L.weights(), s_gpu, w_ref, s_ref, G, A, wl.lr)
        # the next step starts, on both sides, from the state the GPU reached
        L.w_host = L.weights().copy()
        L.s_host = s_gpu.copy()


@pytest.mark.parametrize("shape", ["rowhash-2M", "z64-two-chunks", "multihot-z64"])
def test_runs_deterministic(shape):
    """The same update from the same state twice: bit-identical weights and
    states (no float atomics; run sums and tile sums in a fixed order)."""
    results = []
    for _ in range(2):
        L = _layer(shape, wl=dict(optimizer="adagrad", lr=0.01), s0=0.1)
        L.backward(synth.make_grad(L.wl, L.B, batch=0))
        results.append((L.weights().copy(), L.state.cpu().numpy().copy()))
    assert np.array_equal(results[0][0].view(np.uint8), results[1][0].view(np.uint8))
    assert np.array_equal(results[0][1].view(np.uint32), results[1][1].view(np.uint32))
