"""PSS_PREPARE_BACKWARD: the forward groups the batch for the next backward on
the same stream, on a library stream, or (when it runs the streamed kernel)
by writing the grouping's keygen stage itself.  Every result is checked
against the oracle, including the cases where the prepared grouping must not
be used."""
import numpy as np
import pytest
import torch

import synth
from synth.gen import Inputs
from paper_2207_10731_amd import pss
import parity
from parity import Layer

pytestmark = pytest.mark.gpu

PREP = pss.PSS_PREPARE_BACKWARD


def _check_forward(L, got):
    ref, s_abs = L.ref_forward()
    parity.check_forward(got, ref, s_abs, parity.RTOL[L.wl.weight_dtype])


def _check_update(L, g):
    w_ref, s_ref, G, A, _ = L.ref_backward(g)
    s_gpu = None if L.state is None else L.state.cpu().numpy()
    parity.check_update(L, L.weights(), s_gpu, w_ref, s_ref, G, A, L.wl.lr)


@pytest.mark.parametrize("key,B,kw", [("c2", 700, {}), ("c2", 300, dict(idx32=True)),
                                      ("c3", 50, dict(mean=True)), ("c1", None, {})],
                         ids=["onehot", "onehot-i32", "multihot-mean", "tiny"])
def test_prepared_step(key, B, kw):
    L = Layer(synth.get(key), B=B, flags=pss.PSS_BWD_SORTED | PREP, **kw)
    g = synth.make_grad(L.wl, B=L.B)
    _check_forward(L, L.forward())
    L.backward(g)
    _check_update(L, g)


def test_prepared_for_other_indices_is_not_used():
    """Prepared for batch A, then a backward of batch B (same shapes) on the
    same stream, then a backward of A: both are computed from their own
    indices."""
    A = Layer(synth.get("c2"), B=700, batch=0, flags=PREP)
    Bl = Layer(synth.get("c2"), B=700, batch=1, flags=PREP)
    gA = synth.make_grad(A.wl, B=A.B, batch=0)
    gB = synth.make_grad(Bl.wl, B=Bl.B, batch=1)
    A.forward()
    Bl.backward(gB)
    _check_update(Bl, gB)
    A.backward(gA)
    _check_update(A, gA)


def test_two_forwards_then_two_backwards():
    """Only the last forward's grouping is kept: the first backward groups
    its batch itself, the second reuses the prepared one."""
    A = Layer(synth.get("c2"), B=700, batch=0, flags=PREP)
    Bl = Layer(synth.get("c2"), B=700, batch=1, flags=PREP)
    gA = synth.make_grad(A.wl, B=A.B, batch=0)
    gB = synth.make_grad(Bl.wl, B=Bl.B, batch=1)
    A.forward()
    Bl.forward()
    A.backward(gA)
    Bl.backward(gB)
    _check_update(A, gA)
    _check_update(Bl, gB)


def test_repeated_steps_reuse_the_buffer():
    """Several prepared steps in a row on one stream (weights updated in
    place each step), against the oracle applied step by step."""
    L = Layer(synth.get("c2"), B=400, flags=PREP)
    w = L.w_host.copy()
    for k in range(3):
        g = synth.make_grad(L.wl, B=L.B, batch=k)
        L.w_host = w
        L.shared.copy_(torch.from_numpy(w).to(L.dev))
        torch.cuda.synchronize()
        L.forward()
        L.backward(g)
        _check_update(L, g)
        w = L.weights().copy()


def test_prepare_then_release():
    L = Layer(synth.get("c2"), B=300, flags=PREP)
    g = synth.make_grad(L.wl, B=L.B)
    L.forward()
    pss.pss_release_scratch()
    L.backward(g)
    _check_update(L, g)


def test_prepared_step_in_a_graph():
    """Forward with the flag (and the explicit prepare call) and backward
    captured into one graph: under capture both are ignored; three replays from the same weights, with
    eager prepared steps in between, each match the oracle."""
    dev = torch.device("cuda", 0)
    L = Layer(synth.get("c2"), B=300, flags=PREP)
    other = Layer(synth.get("c2"), B=500, batch=1, flags=PREP)
    g = synth.make_grad(L.wl, B=L.B)
    g_other = synth.make_grad(other.wl, B=other.B, batch=1)
    g_dev = torch.from_numpy(g).to(dev)
    w0 = torch.from_numpy(L.w_host).to(dev)
    out = torch.empty((L.B, L.wl.T * L.wl.d), device=dev)
    wl = L.wl
    L.forward()
    L.backward(g)  # eager warm-up outside capture
    L.shared.copy_(w0)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=torch.cuda.Stream()):
        s = torch.cuda.current_stream()
        # the explicit call does nothing while the stream is being captured
        pss.pss_prepare_backward(wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets, stream=s)
        pss.pss_forward(L.shared, wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets, out, stream=s)
        pss.pss_backward_update(L.shared, None, wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets,
                                g_dev, wl.lr, stream=s)
    torch.cuda.synchronize()
    for _ in range(3):
        L.shared.copy_(w0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        _check_update(L, g)
        got = out.cpu().numpy()
        ref, s_abs = L.ref_forward()
        parity.check_forward(got, ref, s_abs, parity.RTOL[wl.weight_dtype])
        other.shared.copy_(torch.from_numpy(other.w_host).to(dev))
        other.forward()
        other.backward(g_other)
        _check_update(other, g_other)
    del graph
    assert np.isfinite(L.weights()).all()


def test_backward_uses_the_grouping_made_by_the_forward():
    """White box: after the forward with the flag (and a synchronisation, so
    its grouping has finished), the indices tensor is overwritten in place
    with another batch's, which the flag forbids.  The backward still
    deposits at the addresses of the batch the forward grouped: it used the
    prepared grouping.  Without the flag the same sequence follows the new
    contents."""
    for flags, grouped_batch in [(PREP, 0), (0, 1)]:
        L = Layer(synth.get("c2"), B=700, batch=0, flags=flags)
        other = synth.make_inputs(L.wl, B=L.B, batch=1)
        g = synth.make_grad(L.wl, B=L.B)
        L.forward()
        L.indices.copy_(torch.from_numpy(other.indices).to(L.dev))
        torch.cuda.synchronize()
        L.backward(g)
        if grouped_batch == 1:
            L.x = other
        _check_update(L, g)


@pytest.mark.parametrize("key,B,kw", [("c2", 700, {}), ("c3", 50, dict(mean=True))],
                         ids=["onehot", "multihot-mean"])
def test_explicit_prepare_call(key, B, kw):
    """pss_prepare_backward, then a forward without the flag, then the
    backward: the same results as without any preparation."""
    L = Layer(synth.get(key), B=B, **kw)
    wl = L.wl
    g = synth.make_grad(wl, B=L.B)
    pss.pss_prepare_backward(wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets)
    _check_forward(L, L.forward())
    L.backward(g)
    _check_update(L, g)


def test_explicit_prepare_is_used_by_the_backward():
    """White box, as for the flag: after pss_prepare_backward (and a
    synchronisation) the indices are overwritten in place with another
    batch's, which the contract forbids; the backward still deposits at the
    addresses of the batch that was grouped."""
    L = Layer(synth.get("c2"), B=700, batch=0)
    wl = L.wl
    other = synth.make_inputs(wl, B=L.B, batch=1)
    g = synth.make_grad(wl, B=L.B)
    pss.pss_prepare_backward(wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets)
    torch.cuda.synchronize()
    L.indices.copy_(torch.from_numpy(other.indices).to(L.dev))
    torch.cuda.synchronize()
    L.backward(g)
    _check_update(L, g)  # the oracle still sees batch 0


def test_prepared_on_two_streams():
    """Groupings prepared on two streams at once for two batches: each
    stream's backward reuses its own, and both match the oracle."""
    dev = torch.device("cuda", 0)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    Ls = [Layer(synth.get("c2"), B=700, batch=k) for k in range(2)]
    gs = [synth.make_grad(L.wl, B=L.B, batch=k) for k, L in enumerate(Ls)]
    gd = [torch.from_numpy(g).to(dev) for g in gs]
    outs = [torch.empty((L.B, L.wl.T * L.wl.d), device=dev) for L in Ls]
    torch.cuda.synchronize()
    for L, s in zip(Ls, streams):
        wl = L.wl
        pss.pss_prepare_backward(wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets, stream=s)
    for L, s, out, g in zip(Ls, streams, outs, gd):
        wl = L.wl
        pss.pss_forward(L.shared, wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets, out, stream=s)
        pss.pss_backward_update(L.shared, None, wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets, g,
                                wl.lr, stream=s)
    torch.cuda.synchronize()
    for L, out, g in zip(Ls, outs, gs):
        _check_forward(L, out.cpu().numpy())
        _check_update(L, g)



# The streamed forward (one item per bag, d in {64, 128, 256}, Z % 4 == 0,
# array within the aggregate L2) writes the keygen stage of the grouping; the
# backward finishes it.  Shapes: the XCD groups' share of the sort tiles,
# ragged last tiles, a grid too small for the XCD groups.
FUSED = {
    "c2-700": dict(key="c2", B=700),
    "c2-4000": dict(key="c2", B=4000),        # 51 sort tiles over 8 XCD groups
    "d64-t7": dict(key="c2", B=1001, T=7, d=64, Z=16, M=1_000_000),
    "small-grid": dict(key="c2", B=20, T=2, M=50_000),
}


def _fused_layer(case, **kw):
    c = dict(FUSED[case])
    wl = synth.get(c.pop("key"))
    B = c.pop("B")
    if c:
        wl = wl.scaled(**c)
    return Layer(wl, B=B, **kw)


@pytest.mark.parametrize("case", list(FUSED))
@pytest.mark.parametrize("opt", ["plain", "i32", "mean", "sign"])
def test_fused_keygen_step(case, opt):
    kw = {"plain": {}, "i32": dict(idx32=True), "mean": dict(mean=True),
          "sign": dict(sign="sparse")}[opt]
    print(f"fused keygen case {case} {opt}", flush=True)
    L = _fused_layer(case, flags=pss.PSS_BWD_SORTED | PREP, **kw)
    g = synth.make_grad(L.wl, B=L.B)
    _check_forward(L, L.forward())
    L.backward(g)
    _check_update(L, g)


def _irregular(T, B, seed, k, n_index=50_000):
    """N == T*B items, but k empty bags and k bags of two items: the
    streamed forward's slow path, and the keygen's bag search."""
    rng = np.random.default_rng(seed)
    pick = rng.permutation(T * B)
    lengths = np.ones(T * B, dtype=np.int64)
    lengths[pick[:k]] = 0
    lengths[pick[k:2 * k]] = 2
    offsets = np.zeros(T * B + 1, dtype=np.int64)
    np.cumsum(lengths, out=offsets[1:])
    indices = rng.integers(0, n_index, size=int(offsets[-1]), dtype=np.int64)
    return indices, offsets


@pytest.mark.parametrize("mean", [False, True])
def test_fused_keygen_irregular_bags(mean):
    """As many items as bags but not one per bag: the forward still streams
    and writes the keygen stage, whose items search their bags."""
    wl = synth.get("c2").scaled(T=6, M=700_000)
    L = Layer(wl, B=900, flags=pss.PSS_BWD_SORTED | PREP, mean=mean)
    indices, offsets = _irregular(wl.T, L.B, 5, 300)
    L.x = Inputs(indices=indices, offsets=offsets, B=L.B)
    L.indices = torch.from_numpy(indices).to(L.dev)
    L.offsets = torch.from_numpy(offsets).to(L.dev)
    g = synth.make_grad(wl, B=L.B)
    _check_forward(L, L.forward())
    L.backward(g)
    _check_update(L, g)


def test_fused_keygen_bf16_storage_and_adagrad():
    """The fused stage serves the backward whatever the update: bf16 storage
    with SGD (G buffer and optimizer pass), and Adagrad."""
    wl = synth.get("c2").scaled(T=8, M=1_000_000)
    for w in (wl.scaled(weight_dtype="bf16"), wl.scaled(optimizer="adagrad", lr=0.01)):
        L = Layer(w, B=600, flags=pss.PSS_BWD_SORTED | PREP, s0=0.1)
        g = synth.make_grad(w, B=L.B)
        _check_forward(L, L.forward())
        L.backward(g)
        _check_update(L, g)


def test_fused_keygen_run_sums_by_address():
    """Whole-row chunks with the deposit by address (run sums by address):
    the backward finishes the fused grouping, then deposits by address."""
    wl = synth.get("c2").scaled(T=5, Z=128, M=300_000)
    L = Layer(wl, B=800, flags=pss.PSS_BWD_SORTED | PREP | pss.PSS_DEPOSIT_BY_ADDRESS)
    g = synth.make_grad(wl, B=L.B)
    _check_forward(L, L.forward())
    L.backward(g)
    _check_update(L, g)


def test_fused_keygen_after_explicit_prepare():
    """pss_prepare_backward (library stream), then the forward with the flag
    for the same batch (its keygen replaces the library stream's grouping,
    after waiting for it), then the backward."""
    L = _fused_layer("c2-700", flags=PREP)
    wl = L.wl
    g = synth.make_grad(wl, B=L.B)
    pss.pss_prepare_backward(wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets)
    _check_forward(L, L.forward())
    L.backward(g)
    _check_update(L, g)
    # and the other way round: a fused stage left unused, then an explicit
    # preparation and a forward without the flag
    M2 = Layer(wl, B=L.B, batch=1)
    g2 = synth.make_grad(wl, B=M2.B, batch=1)
    L.forward()
    pss.pss_prepare_backward(wl.M, wl.Z, wl.d, M2.hp, M2.indices, M2.offsets)
    _check_forward(M2, M2.forward())
    M2.backward(g2)
    _check_update(M2, g2)
