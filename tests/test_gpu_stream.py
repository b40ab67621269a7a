"""GPU parity of the streamed forward (batches with as many items as bags,
Z % 4 == 0, d in {64, 128, 256}, shared array within the aggregate L2) against
the oracle (Sec. 2.4 forward, Sec. 2.5 mapping).

One-hot bags copy a chunk's weights (times a sign, or divided by a bag length
of 1), so those outputs must equal the oracle bit for bit.  Cases cover every
row-piece count per 1 KB unit (d = 64, 128, 256), chunk sizes from 4 to d, a
ragged last unit, chunks that wrap past the end of the array (small M, and
M = Z where nearly every chunk wraps), both sign modes, mean pooling, int32
indices, bfloat16 storage and rows, batches too small to fill one wavefront
per unit, and batches whose bags are not all single items (empty bags, bags of
two items, items stored out of bag order), which take the slow path.
The grid's XCD groups each own a share of the tables, in periods of L rows
(T*L divisible by the group count): table counts with L = 1, 2, 4 and 8,
batches whose last period is ragged, and a grid too small for the groups
(one group in row order) are covered.
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

C2 = synth.get("c2")


def _wl(T, B, d, Z, M, dtype="f32", card="fixed:100000", dist="zipf:1.1"):
    return C2.scaled(T=T, B=B, d=d, Z=Z, M=M, weight_dtype=dtype, cardinality=card, index_dist=dist)


# (T, B, d, Z, M): all one-hot
SHAPES = {
    "d128z32": (26, 700, 128, 32, 2_500_000),
    "d128z4": (5, 333, 128, 4, 100_000),
    "d128z128": (3, 257, 128, 128, 50_000),
    "d64z16": (7, 333, 64, 16, 1_000_000),      # 2331 pieces: ragged last unit
    "d64z64": (1, 5, 64, 64, 4096),             # 5 pieces: fewer units than wavefronts
    "d256z8": (4, 301, 256, 8, 700_000),
    "d256z256": (2, 129, 256, 256, 300_000),
    "wrap4096": (6, 400, 128, 32, 4096),        # base + 31 >= M for ~0.8% of chunks
    "wrapMZ": (3, 200, 128, 128, 128),          # M = Z: almost every chunk wraps
    "wrapM260": (2, 300, 64, 64, 260),
    # how the tables are shared among the 8 XCD groups: periods of L rows
    # with T*L divisible by 8 (L = 1, 2, 4, 8), B not a multiple of L
    "T8": (8, 301, 128, 32, 1_000_000),         # L = 1
    "T26odd": (26, 701, 128, 32, 2_500_000),    # L = 4, ragged last period
    "T12": (12, 333, 64, 32, 500_000),          # L = 2
    "nx1": (2, 20, 128, 32, 50_000),            # 5 workgroups: one group, row order
}


@pytest.mark.parametrize("shape", list(SHAPES))
def test_stream_forward_one_hot_bit_exact(shape):
    T, B, d, Z, M = SHAPES[shape]
    print(f"stream case {shape}: T={T} B={B} d={d} Z={Z} M={M}", flush=True)
    L = Layer(_wl(T, B, d, Z, M))
    got = L.forward()
    ref, _ = L.ref_forward()
    assert np.array_equal(got.astype(np.float64), ref)


OPTS = {
    "pm1": dict(sign="pm1"),
    "sparse": dict(sign="sparse"),
    "mean": dict(mean=True),
    "i32": dict(idx32=True),
    "all": dict(sign="sparse", mean=True, idx32=True),
}


@pytest.mark.parametrize("opt", list(OPTS))
@pytest.mark.parametrize("shape", ["d64z16", "d128z32", "d256z8", "wrap4096"])
def test_stream_forward_options_bit_exact(shape, opt):
    T, B, d, Z, M = SHAPES[shape]
    print(f"stream case {shape} opts {opt}", flush=True)
    L = Layer(_wl(T, B, d, Z, M), **OPTS[opt])
    got = L.forward()
    ref, _ = L.ref_forward()
    assert np.array_equal(got.astype(np.float64), ref)


@pytest.mark.parametrize("shape", ["d128z32", "d64z16", "wrap4096"])
def test_stream_forward_bf16(shape):
    """bfloat16 storage (widened exactly: bit-exact) and bfloat16 rows (one
    rounding of the exact float32 copy: equal to torch's rounding)."""
    T, B, d, Z, M = SHAPES[shape]
    print(f"stream case {shape} bf16", flush=True)
    L = Layer(_wl(T, B, d, Z, M, dtype="bf16"))
    got = L.forward()
    ref, _ = L.ref_forward()
    assert np.array_equal(got.astype(np.float64), ref)
    L = Layer(_wl(T, B, d, Z, M), rows_bf16=True)
    got = L.forward()
    ref, _ = L.ref_forward()
    want = torch.from_numpy(ref.astype(np.float32)).to(torch.bfloat16).float().numpy()
    assert np.array_equal(got, want)


def _irregular(T, B, seed, k):
    """N == T*B items, but k empty bags and k bags of two items."""
    rng = np.random.default_rng(seed)
    pick = rng.permutation(T * B)
    lengths = np.ones(T * B, dtype=np.int64)
    lengths[pick[:k]] = 0
    lengths[pick[k:2 * k]] = 2
    offsets = np.zeros(T * B + 1, dtype=np.int64)
    np.cumsum(lengths, out=offsets[1:])
    indices = rng.integers(0, 50_000, size=int(offsets[-1]), dtype=np.int64)
    return indices, offsets


@pytest.mark.parametrize("mean", [False, True])
@pytest.mark.parametrize("shape", ["d128z32", "d64z16", "d256z8", "wrap4096"])
def test_stream_forward_slow_path(shape, mean):
    """Bags that are not a single item at position g (empty, two items, and the
    one-item bags after them, whose item sits at another position) are pooled
    by the slow path; the batch still has as many items as bags."""
    T, B, d, Z, M = SHAPES[shape]
    print(f"stream slow-path case {shape} mean={mean}", flush=True)
    wl = _wl(T, B, d, Z, M)
    indices, offsets = _irregular(T, B, 7, 40)
    assert indices.shape[0] == T * B
    dev = torch.device("cuda", 0)
    w = synth.make_weights(wl)
    a, b = o.hash_params_from_seed(wl.hash_seed)
    hp = pss.make_hash_params(wl.hash_seed, num_tables=T, batch=B, num_indices=T * B,
                              flags=pss.PSS_POOL_MEAN if mean else 0)
    out = torch.empty((B, T * d), dtype=torch.float32, device=dev)
    pss.pss_forward(torch.from_numpy(w).to(dev), M, Z, d, hp, torch.from_numpy(indices).to(dev),
                    torch.from_numpy(offsets).to(dev), out)
    torch.cuda.synchronize()
    ref, s_abs = o.forward64(w, M, Z, d, T, B, a, b, indices, offsets, mean=mean)
    parity.check_forward(out.cpu().numpy(), ref, s_abs, 1e-5)
    # every bag of one item is still an exact copy
    lengths = np.diff(offsets).reshape(T, B).T.repeat(d, axis=1)
    one = lengths == 1
    assert np.array_equal(out.cpu().numpy().astype(np.float64)[one], ref[one])


def test_stream_forward_batches_back_to_back():
    """Two forwards on different batches and shapes in a row (the grid size
    follows the batch) each match the oracle."""
    for shape in ["d128z32", "d64z64", "d256z256"]:
        T, B, d, Z, M = SHAPES[shape]
        L = Layer(_wl(T, B, d, Z, M))
        got = L.forward()
        ref, _ = L.ref_forward()
        assert np.array_equal(got.astype(np.float64), ref)
