"""GPU parity of the layer's options against the oracle: chunk signs from a
second universal hash (Sec. 2.5, Achlioptas-type entries: +-1, or +-1/0),
mean pooling, int32 indices/offsets and bfloat16 pooled rows, on the dense
(atomic, sorted) and sparse backward variants."""
import numpy as np
import pytest
import torch

import synth
from oracle import pss_oracle as o
from paper_2207_10731_amd import pss
import parity
from parity import Layer

pytestmark = pytest.mark.gpu

# (workload, batch, M override): multi-item bags with a lookup table of bases
# (c3, C = 4), one-hot bags (c2), many chunks per row without the table (c4,
# C = 128), bf16 storage with whole-row chunks (c5), and a tiny layout with
# empty and long bags (c1 with Poisson(12) lengths in [0, 64]).
CASES = {
    "c1pois": (synth.get("c1").scaled(bag="poisson:12:0:64", B=300), None, None),
    "c2": (synth.get("c2"), 700, None),
    "c3": (synth.get("c3"), 50, None),
    "c4": (synth.get("c4"), 200, 50_000_000),
    "c5": (synth.get("c5"), 600, None),
}
OPTS = {
    "pm1": dict(sign="pm1"),
    "sparse": dict(sign="sparse"),
    "mean": dict(mean=True),
    "i32": dict(idx32=True),
    "bf16rows": dict(rows_bf16=True),
    "all": dict(sign="sparse", mean=True, idx32=True, rows_bf16=True),
    "pm1-mean-bf16": dict(sign="pm1", mean=True, rows_bf16=True),
}
VARIANTS = {"atomic": pss.PSS_BWD_ATOMIC, "sorted": pss.PSS_BWD_SORTED,
            "sparse": pss.PSS_BWD_SPARSE}


def _layer(case, flags=pss.PSS_BWD_AUTO, **opts):
    wl, B, M = CASES[case]
    print(f"options case={case} B={B} M={M} flags={flags} opts={opts}", flush=True)
    return Layer(wl, B=B, M=M, flags=flags, **opts)


@pytest.mark.parametrize("mode", ["pm1", "sparse"])
@pytest.mark.parametrize("case", ["c1pois", "c3", "c4"])
def test_sign_factors_bit_exact(case, mode):
    L = _layer(case, sign=mode)
    got = L.debug_signs()
    _, t, _ = o.item_bags(L.wl.T, L.B, L.x.offsets)
    want = o.signs_for(L.wl.Z, L.wl.d, L.wl.T, L.sign[1], L.sign[2], L.x.indices, t, mode)
    assert np.array_equal(got.astype(np.int64), want)


@pytest.mark.parametrize("opt", list(OPTS))
@pytest.mark.parametrize("case", list(CASES))
def test_forward_options(case, opt):
    L = _layer(case, **OPTS[opt])
    got = L.forward()
    ref, s_abs = L.ref_forward()
    parity.check_forward(got, ref, s_abs, 1e-5, rows_bf16=L.rows_bf16)


@pytest.mark.parametrize("variant", list(VARIANTS))
@pytest.mark.parametrize("opt", list(OPTS))
@pytest.mark.parametrize("case", ["c1pois", "c3", "c4", "c5"])
def test_backward_options(case, opt, variant):
    L = _layer(case, flags=VARIANTS[variant], **OPTS[opt])
    grad = synth.make_grad(L.wl, L.B, batch=0)
    L.backward(grad)
    w_ref, s_ref, G, A, _ = L.ref_backward(grad)
    s_gpu = None if L.state is None else L.state.cpu().numpy()
    parity.check_update(L, L.weights(), s_gpu, w_ref, s_ref, G, A, L.wl.lr)


def test_forward_integer_valued_with_signs_bit_exact():
    """w[m] = m with +-1/0 factors: every pooled value is an integer below
    2^24 in magnitude, so the GPU must match the oracle bit for bit."""
    wl = synth.get("c1").scaled(B=200, bag="poisson:12:0:64")
    w = np.arange(wl.M, dtype=np.float32)
    for sign in ("pm1", "sparse"):
        L = Layer(wl, w=w, sign=sign)
        got = L.forward()
        want = o.forward(w, wl.M, wl.Z, wl.d, wl.T, L.B, L.a, L.b, L.x.indices, L.x.offsets,
                         sign=L.sign)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("opt", ["sparse", "all", "mean"])
@pytest.mark.parametrize("case", ["c1pois", "c3", "c4"])
def test_sparse_gradient_options(case, opt):
    """Unique locations bit-exact (chunks of factor 0 are not locations) and
    summed values within tolerance."""
    L = _layer(case, **OPTS[opt])
    wl = L.wl
    grad = synth.make_grad(wl, L.B, batch=0)
    g = torch.from_numpy(grad)
    if L.rows_bf16:
        g = g.to(torch.bfloat16)
    g = g.to(L.dev)
    cap = min(wl.M, L.x.N * wl.d)
    loc = torch.empty(cap, dtype=torch.int32, device=L.dev)
    val = torch.empty(cap, dtype=torch.float32, device=L.dev)
    cnt = torch.zeros(1, dtype=torch.int64, device=L.dev)
    pss.pss_gradient_sparse(wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets, g, loc, val, cnt)
    torch.cuda.synchronize()
    n = int(cnt.item())
    got_loc = loc[:n].cpu().numpy().view(np.uint32).astype(np.int64)
    want_loc, want_val = o.gradient_sparse(wl.M, wl.Z, wl.d, wl.T, L.B, L.a, L.b, L.x.indices,
                                           L.x.offsets, L.grad_values(grad), sign=L.sign,
                                           mean=L.mean)
    assert np.array_equal(got_loc, want_loc)
    _, A, _ = o.gradient_dense(wl.M, wl.Z, wl.d, wl.T, L.B, L.a, L.b, L.x.indices, L.x.offsets,
                               L.grad_values(grad), sign=L.sign, mean=L.mean)
    err = np.abs(val[:n].cpu().numpy().astype(np.float64) - want_val)
    assert np.all(err <= 1e-5 * A[want_loc] + 1e-30)


@pytest.mark.parametrize("case", ["c1pois", "c3"])
def test_int32_indices_give_identical_bits(case):
    """int32 and int64 index arrays describe the same lookups: forward rows
    and the (deterministic) sparse backward update agree bit for bit."""
    outs, ws = [], []
    for idx32 in (False, True):
        L = _layer(case, flags=pss.PSS_BWD_SPARSE, idx32=idx32, sign="pm1")
        outs.append(L.forward())
        L.backward(synth.make_grad(L.wl, L.B, batch=0))
        ws.append(L.weights())
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
    assert np.array_equal(ws[0].view(np.uint32), ws[1].view(np.uint32))


def test_compress_with_signs_matches_oracle():
    """Post-hoc M = S E with signed S (Thm. 2 with the +-1 entries of
    Sec. 2.5) and its retrieval."""
    T, n, d, Z, M = 2, 1500, 64, 16, 9001
    E = np.random.default_rng(2).standard_normal((T, n, d)).astype(np.float32)
    for flag, mode in ((pss.PSS_SIGN_PM1, "pm1"), (pss.PSS_SIGN_SPARSE, "sparse")):
        hp = pss.make_hash_params(6, num_tables=T, batch=n, num_indices=T * n, flags=flag)
        sign = (mode, hp.sign_a, hp.sign_b)
        shared = pss.compress_table(torch.from_numpy(E).cuda(), M, Z, hp)
        got = shared.cpu().numpy().astype(np.float64)
        idx = np.tile(np.arange(n, dtype=np.int64), T)
        off = np.arange(T * n + 1, dtype=np.int64)
        grad = E.transpose(1, 0, 2).reshape(n, T * d)
        G, A, _ = o.gradient_dense(M, Z, d, T, n, hp.a, hp.b, idx, off, grad, sign=sign)
        assert np.all(np.abs(got - G) <= 1e-5 * A + 1e-30)
        R = pss.lookup_rows(shared, M, Z, d, T, n, hp).cpu().numpy()
        want, _ = o.forward64(got.astype(np.float32), M, Z, d, T, n, hp.a, hp.b, idx, off,
                              sign=sign)
        assert np.array_equal(R.astype(np.float64), want.reshape(n, T, d).transpose(1, 0, 2))
