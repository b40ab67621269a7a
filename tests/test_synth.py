"""Seeded input generators and the oracle's sampled helpers (no GPU)."""
import numpy as np
import pytest

import synth
from synth import gen
from oracle import pss_oracle as o


@pytest.mark.parametrize("key", ["c1", "c2", "c3", "c4", "c5"])
def test_inputs_shapes_and_determinism(key):
    wl = synth.get(key)
    B = 64
    x1 = synth.make_inputs(wl, B=B)
    x2 = synth.make_inputs(wl, B=B)
    assert np.array_equal(x1.indices, x2.indices) and np.array_equal(x1.offsets, x2.offsets)
    assert x1.offsets.shape == (wl.T * B + 1,) and x1.offsets[0] == 0
    assert x1.offsets[-1] == x1.N and np.all(np.diff(x1.offsets) >= 0)
    card = gen.cardinalities(wl)
    t_of = np.repeat(np.arange(wl.T * B) // B, np.diff(x1.offsets))
    assert np.all(x1.indices >= 0) and np.all(x1.indices < card[t_of])
    lens = np.diff(x1.offsets)
    if wl.bag == "one":
        assert np.all(lens == 1)
    else:
        assert lens.min() >= 1 and lens.max() <= 64 and 15 < lens.mean() < 25
    other = synth.make_inputs(wl, B=B, batch=1)
    assert not np.array_equal(other.indices, x1.indices)
    g = synth.make_grad(wl, B=B)
    assert g.shape == (B, wl.T * wl.d) and g.dtype == np.float32
    assert np.array_equal(g, synth.make_grad(wl, B=B))
    o.validate(wl.M, wl.Z, wl.d, wl.T, B, 1, 0, x1.indices, x1.offsets, wl.weight_dtype)


def test_cardinalities_criteo_shaped():
    card = gen.cardinalities(synth.get("c2"))
    assert card.shape == (26,) and card.min() >= 3 and card.max() <= 40_000_000
    assert card.max() > 100 * card.min()


def test_weights_and_bf16_storage():
    wl = synth.get("c1")
    w = synth.make_weights(wl, M=1000)
    assert w.dtype == np.float32 and np.all(np.abs(w) <= 0.01)
    wb = synth.make_weights(synth.get("c5"), M=1000)
    assert wb.dtype == np.uint16
    assert np.all(np.abs(o.widen(wb, "bf16")) <= 0.0101)


def test_zipf_is_skewed_and_truncated():
    rng = np.random.default_rng(0)
    r = gen._zipf_truncated(rng, 1.1, 5, 20000)
    assert r.min() >= 0 and r.max() <= 4
    counts = np.bincount(r, minlength=5)
    assert np.all(np.diff(counts) < 0)


def test_sampled_helpers_match_full_oracle():
    wl = synth.get("c3").scaled(M=20011)
    B = 48
    x = synth.make_inputs(wl, B=B)
    a, b = o.hash_params_from_seed(wl.hash_seed)
    w = synth.make_weights(wl)
    g = synth.make_grad(wl, B=B)
    out, sabs = o.forward64(w, wl.M, wl.Z, wl.d, wl.T, B, a, b, x.indices, x.offsets)
    bags = np.array([0, 5, wl.T * B - 1, 77])
    part, psabs = o.forward_at(w, wl.M, wl.Z, wl.d, wl.T, B, a, b, x.indices, x.offsets, bags)
    for r, gg in enumerate(bags):
        t, bb = divmod(int(gg), B)
        np.testing.assert_allclose(part[r], out[bb, t * wl.d:(t + 1) * wl.d], rtol=1e-12)
        np.testing.assert_allclose(psabs[r], sabs[bb, t * wl.d:(t + 1) * wl.d], rtol=1e-12)
    G, A, cnt = o.gradient_dense(wl.M, wl.Z, wl.d, wl.T, B, a, b, x.indices, x.offsets, g)
    where = np.random.default_rng(1).choice(wl.M, 300, replace=False)
    Gs, As, cs = o.gradient_at(wl.M, wl.Z, wl.d, wl.T, B, a, b, x.indices, x.offsets, g, where)
    np.testing.assert_allclose(Gs, G[where], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(As, A[where], rtol=1e-10, atol=1e-12)
    assert np.array_equal(cs, cnt[where])


def test_validate_rejects_bad_arguments():
    off = np.array([0, 1], dtype=np.int64)
    idx = np.array([3], dtype=np.int64)
    ok = dict(M=100, Z=4, d=8, T=1, B=1, a=5, b=0, indices=idx, offsets=off)
    o.validate(**ok)
    for bad in [dict(M=0), dict(M=2**31), dict(Z=0), dict(Z=3), dict(d=4097), dict(a=0),
                dict(a=2**31 - 1), dict(b=2**31 - 1), dict(B=0),
                dict(offsets=np.array([0, 2])), dict(indices=np.array([-1])),
                dict(indices=np.array([2**31]))]:
        with pytest.raises(ValueError):
            o.validate(**{**ok, **bad})
    with pytest.raises(ValueError):
        o.validate(**ok, weight_dtype="f16")
