"""The binding refuses tensors shorter than the sizes a call declares (the
kernels trust M, N, T*B and d) and tensors on another device, before
anything is enqueued; a call with exact sizes still matches the oracle."""
import pytest
import torch

import synth
from paper_2207_10731_amd import pss
import parity
from parity import Layer

pytestmark = pytest.mark.gpu


def _args(L):
    wl = L.wl
    out = torch.empty((L.B, wl.T * wl.d), device=L.dev)
    g = torch.from_numpy(synth.make_grad(wl, B=L.B)).to(L.dev)
    return wl, out, g


def test_short_tensors_are_refused():
    L = Layer(synth.get("c1"))
    wl, out, g = _args(L)
    fwd = dict(shared=L.shared, indices=L.indices, offsets=L.offsets, out=out)
    for name in fwd:
        bad = dict(fwd)
        bad[name] = fwd[name][:-1]
        with pytest.raises(ValueError):
            pss.pss_forward(bad["shared"], wl.M, wl.Z, wl.d, L.hp, bad["indices"],
                            bad["offsets"], bad["out"])
    state = torch.zeros(wl.M, device=L.dev)
    bwd = dict(shared=L.shared, state=state, indices=L.indices, offsets=L.offsets, grad=g)
    for name in bwd:
        bad = dict(bwd)
        bad[name] = bwd[name].reshape(-1)[:-1]
        with pytest.raises(ValueError):
            pss.pss_backward_update(bad["shared"], bad["state"], wl.M, wl.Z, wl.d, L.hp,
                                    bad["indices"], bad["offsets"], bad["grad"], wl.lr)
    base = torch.empty(L.x.indices.size * (wl.d // wl.Z) - 1, dtype=torch.int32, device=L.dev)
    with pytest.raises(ValueError):
        pss.pss_debug_addresses(wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets, base)
    torch.cuda.synchronize()
    # nothing was enqueued: the array is untouched, and an exact call works
    assert (L.weights() == L.w_host).all()
    got = pss.pss_forward(L.shared, wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets, out)
    ref, s_abs = L.ref_forward()
    parity.check_forward(got.cpu().numpy(), ref, s_abs, parity.RTOL[wl.weight_dtype])


def test_reduce_events_hook_brackets_the_reduce_kernel():
    """With the timing hook set, the dispatch of a sorted backward's
    reduce-and-deposit kernel records both events at the kernel's start and
    end (a positive interval, inside the call's own); the update made with
    the hook matches the oracle."""
    wl = synth.get("c2").scaled(B=512)
    g = synth.make_grad(wl, B=512)
    L = Layer(wl, flags=pss.PSS_BWD_SORTED)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for ev in evs:
        ev.record()  # creates the HIP events
    torch.cuda.synchronize()
    pss.pss_debug_reduce_events(evs[1], evs[2])
    evs[0].record()
    try:
        L.backward(g)
    finally:
        pss.pss_debug_reduce_events()
    evs[3].record()
    torch.cuda.synchronize()
    inner, outer = evs[1].elapsed_time(evs[2]), evs[0].elapsed_time(evs[3])
    print(f"reduce {inner * 1e3:.1f} us of {outer * 1e3:.1f} us", flush=True)
    assert 0.0 < inner < outer
    assert evs[0].elapsed_time(evs[1]) > 0.0 and evs[2].elapsed_time(evs[3]) > 0.0
    w_ref, s_ref, G, A, _ = L.ref_backward(g)
    parity.check_update(L, L.weights(), None, w_ref, s_ref, G, A, wl.lr)
