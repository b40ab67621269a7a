"""Scratch kept per (device, stream) between backward calls: growth on one
stream, calls on two streams at once, release, and calls captured into a
graph (which take their scratch from the pool instead).  Every result is
checked against the oracle."""
import numpy as np
import pytest
import torch

import synth
from paper_2207_10731_amd import pss
import parity
from parity import Layer

pytestmark = pytest.mark.gpu


def _check(L, g):
    w_ref, s_ref, G, A, _ = L.ref_backward(g)
    s_gpu = None if L.state is None else L.state.cpu().numpy()
    parity.check_update(L, L.weights(), s_gpu, w_ref, s_ref, G, A, L.wl.lr)


def _launch_backward(L, g_dev, stream):
    wl = L.wl
    pss.pss_backward_update(L.shared, L.state, wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets, g_dev,
                            wl.lr, stream=stream)


@pytest.mark.parametrize("variant", [pss.PSS_BWD_SORTED, pss.PSS_BWD_SPARSE])
def test_scratch_grows_and_serves_smaller_calls(variant):
    """Small, large, then small again on one stream: the kept buffer grows
    once and the smaller call reuses it."""
    pss.pss_release_scratch()
    for key, B in [("c2", 100), ("c2", 700), ("c3", 50), ("c2", 100)]:
        L = Layer(synth.get(key), B=B, flags=variant)
        g = synth.make_grad(L.wl, B=L.B)
        L.backward(g)
        _check(L, g)


def test_two_streams_at_once():
    """Backward calls enqueued on two streams without a synchronisation in
    between each get their own scratch."""
    dev = torch.device("cuda", 0)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    L1 = Layer(synth.get("c2"), B=700, batch=0)
    L2 = Layer(synth.get("c2"), B=700, batch=1)
    g1 = synth.make_grad(L1.wl, B=L1.B, batch=0)
    g2 = synth.make_grad(L2.wl, B=L2.B, batch=1)
    d1, d2 = torch.from_numpy(g1).to(dev), torch.from_numpy(g2).to(dev)
    torch.cuda.synchronize()
    for _ in range(2):  # the second round reuses both kept buffers
        L1.shared.copy_(torch.from_numpy(L1.w_host).to(dev))
        L2.shared.copy_(torch.from_numpy(L2.w_host).to(dev))
        torch.cuda.synchronize()
        _launch_backward(L1, d1, s1)
        _launch_backward(L2, d2, s2)
        torch.cuda.synchronize()
        _check(L1, g1)
        _check(L2, g2)


def test_release_then_call():
    L = Layer(synth.get("c2"), B=300)
    g = synth.make_grad(L.wl, B=L.B)
    L.backward(g)
    pss.pss_release_scratch()
    pss.pss_release_scratch()  # nothing kept: still fine
    L2 = Layer(synth.get("c2"), B=300)
    L2.backward(g)
    _check(L2, g)


@pytest.mark.parametrize("variant", [pss.PSS_BWD_SORTED, pss.PSS_BWD_SPARSE])
def test_graph_capture_replays(variant):
    """A backward captured into a graph, replayed three times with eager
    library work and synchronisations in between; after each replay (from
    the same starting weights) the update matches the oracle."""
    dev = torch.device("cuda", 0)
    L = Layer(synth.get("c2"), B=300, flags=variant)
    other = Layer(synth.get("c2"), B=700, batch=1)
    g = synth.make_grad(L.wl, B=L.B)
    g_other = synth.make_grad(other.wl, B=other.B, batch=1)
    g_dev = torch.from_numpy(g).to(dev)
    w0 = torch.from_numpy(L.w_host).to(dev)
    # eager call first: the library's pool and kernels are set up outside capture
    L.backward(g)
    L.shared.copy_(w0)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    with torch.cuda.graph(graph, stream=side):
        _launch_backward(L, g_dev, torch.cuda.current_stream())
    torch.cuda.synchronize()
    for r in range(3):
        L.shared.copy_(w0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        _check(L, g)
        # eager work between replays: a backward on the default stream
        other.shared.copy_(torch.from_numpy(other.w_host).to(dev))
        other.backward(g_other)
        _check(other, g_other)
    del graph


def test_threads_on_one_stream():
    """Four host threads enqueue backward calls on the same stream at once;
    each call's kernels stay together in the stream, so the shared scratch
    buffer is never used by two calls at a time."""
    import threading
    dev = torch.device("cuda", 0)
    Ls = [Layer(synth.get("c2"), B=700, batch=k) for k in range(4)]
    gs = [synth.make_grad(L.wl, B=L.B, batch=k) for k, L in enumerate(Ls)]
    ds = [torch.from_numpy(g).to(dev) for g in gs]
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    errors = []

    def work(k):
        try:
            _launch_backward(Ls[k], ds[k], stream)
        except Exception as exc:  # surfaced below
            errors.append(exc)

    threads = [threading.Thread(target=work, args=(k,)) for k in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for L, g in zip(Ls, gs):
        _check(L, g)
