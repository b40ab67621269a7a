"""GPU parity of the address-sorted deposit (PSS_DEPOSIT_BY_ADDRESS: Alg. 1's
scatter_add with the contributions radix-sorted by address tile, summed on
chip per tile and applied once) against the oracle.

Shapes put the array at exactly one tile (2^14 elements), one element past
it, far below it (no sort pass at all), and across thousands of tiles with a
ragged last one; chunk sizes 1 to 32; fused SGD, Adagrad (the gradient
buffer is stored tile by tile) and bfloat16 storage; every option; bags of
several items; and a grad = 1 case whose result is an integer count, equal
bit for bit.  AUTO takes this deposit by itself on the HBM-resident
hashing-trick workload, which test_gpu_fullsize.py checks at full size.
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

ADDR = pss.PSS_BWD_SORTED | pss.PSS_DEPOSIT_BY_ADDRESS
C4 = synth.get("c4")

# name: (workload, B, M, Z)
SHAPES = {
    "z1-50M": (C4, 300, 50_000_000, 1),
    "z1-one-tile": (C4, 40, 16384, 1),
    "z1-tile-plus-one": (C4, 40, 16385, 1),
    "z1-small": (C4, 40, 1000, 1),
    "z4-3M": (C4, 200, 3_000_001, 4),
    "z16-multihot": (synth.get("c3"), 40, 2_000_003, 16),
    "z32-onehot": (synth.get("c2"), 300, 2_500_000, 32),
}


def _layer(shape, **kw):
    wl, B, M, Z = SHAPES[shape]
    wl = wl.scaled(M=M, Z=Z)
    print(f"addr case {shape}: B={B} M={M} Z={Z} {kw}", flush=True)
    return Layer(wl, B=B, flags=kw.pop("flags", ADDR), **kw)


def _check(L, lr=None):
    grad = synth.make_grad(L.wl, L.B, batch=0)
    L.backward(grad, lr=lr)
    w_ref, s_ref, G, A, _ = L.ref_backward(grad, lr=lr)
    s_gpu = None if L.state is None else L.state.cpu().numpy()
    parity.check_update(L, L.weights(), s_gpu, w_ref, s_ref, G, A, L.wl.lr if lr is None else lr)


@pytest.mark.parametrize("shape", list(SHAPES))
def test_addr_update(shape):
    """The workload's own optimizer (SGD, or Adagrad on the multi-hot one)."""
    _check(_layer(shape))


@pytest.mark.parametrize("shape", ["z1-50M", "z1-tile-plus-one", "z16-multihot"])
def test_addr_adagrad(shape):
    wl, B, M, Z = SHAPES[shape]
    L = Layer(wl.scaled(M=M, Z=Z, optimizer="adagrad", lr=0.01), B=B, flags=ADDR, s0=0.1)
    _check(L)


@pytest.mark.parametrize("shape", ["z1-50M", "z4-3M"])
def test_addr_bf16_storage(shape):
    wl, B, M, Z = SHAPES[shape]
    L = Layer(wl.scaled(M=M, Z=Z, weight_dtype="bf16", optimizer="adagrad", lr=0.01), B=B,
              flags=ADDR, s0=0.1)
    _check(L)


OPTS = {
    "pm1": dict(sign="pm1"),
    "sparse": dict(sign="sparse"),
    "mean": dict(mean=True),
    "i32": dict(idx32=True),
    "bf16rows": dict(rows_bf16=True),
    "all": dict(sign="sparse", mean=True, idx32=True, rows_bf16=True),
}


@pytest.mark.parametrize("opt", list(OPTS))
@pytest.mark.parametrize("shape", ["z1-50M", "z16-multihot"])
def test_addr_options(shape, opt):
    _check(_layer(shape, **OPTS[opt]))


@pytest.mark.parametrize("shape", ["z1-50M", "z16-multihot", "z1-small"])
def test_addr_counts_bit_exact(shape):
    """w = 0, grad = 1, lr = 1: every updated weight is minus the number of
    reads of that element, an integer the tile sums reach exactly."""
    wl, B, M, Z = SHAPES[shape]
    wl = wl.scaled(M=M, Z=Z, optimizer="sgd")
    L = Layer(wl, B=B, flags=ADDR, w=np.zeros(M, dtype=np.float32))
    ones = np.ones((B, wl.T * wl.d), dtype=np.float32)
    L.backward(ones, lr=1.0)
    _, _, _, _, cnt = L.ref_backward(ones, lr=1.0)
    got = L.weights()
    assert np.array_equal(got, (-cnt).astype(np.float32))
    # untouched elements keep +0.0 exactly (not -0.0)
    assert not np.signbit(got[cnt == 0]).any()


def test_addr_rejected_with_atomic_or_sparse():
    L = _layer("z1-small")
    for v in (pss.PSS_BWD_ATOMIC, pss.PSS_BWD_SPARSE):
        L.hp.flags = v | pss.PSS_DEPOSIT_BY_ADDRESS
        with pytest.raises(pss.PssError) as ei:
            L.backward(synth.make_grad(L.wl, L.B))
        assert ei.value.status == pss.PSS_ERR_UNSUPPORTED
