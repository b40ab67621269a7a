"""pss_backward_update_noalloc (scratch in the library's static device array,
no allocation) against pss_backward_update, through the C ABI.

Each case runs two calls in a row on the same static array, the second with
a smaller batch, so the second call starts from the first call's leftovers.
Both entry points are also checked against the oracle with the usual
normalised tolerance (Sec. 2.4 backward, Alg. 1); the SPARSE variant sums in
a fixed order, so there the two entry points must agree bit for bit.
"""
import numpy as np
import pytest
import torch

import synth
from paper_2207_10731_amd import pss
import parity
from parity import Layer

pytestmark = pytest.mark.gpu

# (workload, first batch, second batch, M override, variant)
CASES = {
    "sorted-sgd-onehot": ("c2", 900, 300, None, pss.PSS_BWD_SORTED),
    "atomic-sgd-onehot": ("c2", 700, 200, None, pss.PSS_BWD_ATOMIC),
    "sorted-adagrad-multihot": ("c3", 60, 25, 2_000_000, pss.PSS_BWD_SORTED),
    "atomic-adagrad-multihot": ("c3", 60, 25, 2_000_000, pss.PSS_BWD_ATOMIC),
    "sparse-adagrad-multihot": ("c3", 60, 25, 2_000_000, pss.PSS_BWD_SPARSE),
    "auto-bf16-rowhash": ("c5", 500, 150, 1_000_000, pss.PSS_BWD_AUTO),
}


def _pair(key, B, M, variant, batch):
    """Two layers with identical state and inputs: one for each entry point."""
    wl = synth.get(key)
    a = Layer(wl, B=B, M=M, batch=batch, flags=variant, s0=0.1)
    b = Layer(wl, B=B, M=M, batch=batch, flags=variant, s0=0.1)
    return a, b


def _run(L, grad, noalloc):
    wl = L.wl
    g = torch.from_numpy(grad).to(L.dev)
    fn = pss.pss_backward_update_noalloc if noalloc else pss.pss_backward_update
    fn(L.shared, L.state, wl.M, wl.Z, wl.d, L.hp, L.indices, L.offsets, g, wl.lr)
    torch.cuda.synchronize()


@pytest.mark.parametrize("case", list(CASES))
def test_noalloc_matches_backward_update(case):
    key, B1, B2, M, variant = CASES[case]
    for step, B in enumerate((B1, B2)):
        print(f"noalloc case={case} call={step} B={B} M={M} variant={variant}", flush=True)
        ref, got = _pair(key, B, M, variant, batch=step)
        grad = synth.make_grad(ref.wl, B, batch=step)
        _run(ref, grad, noalloc=False)
        _run(got, grad, noalloc=True)
        w_ref, s_ref, G, A, _ = got.ref_backward(grad)
        for L in (ref, got):
            s_gpu = None if L.state is None else L.state.cpu().numpy()
            parity.check_update(L, L.weights(), s_gpu, w_ref, s_ref, G, A, L.wl.lr)
        if variant == pss.PSS_BWD_SPARSE:
            assert np.array_equal(got.weights(), ref.weights())
            assert np.array_equal(got.state.cpu().numpy(), ref.state.cpu().numpy())


def test_noalloc_rejects_more_than_its_scratch():
    """The headline one-hot batch fits (28 MB of grouping); a batch whose
    grouping exceeds the static array is refused before anything runs."""
    wl = synth.get("c2")
    L = Layer(wl, B=700)
    big = pss.make_hash_params(wl.hash_seed, num_tables=wl.T, batch=wl.B * 4,
                               num_indices=wl.T * wl.B * 4)
    w0 = L.shared.clone()
    st = pss.load_library().pss_backward_update_noalloc(
        pss._ptr(L.shared), None, wl.M, wl.Z, wl.d, pss.ctypes.byref(big), pss._ptr(L.indices),
        pss._ptr(L.offsets), pss._ptr(L.shared), pss.ctypes.c_float(0.1), pss._stream(None))
    assert st == pss.PSS_ERR_SCRATCH_LIMIT
    torch.cuda.synchronize()
    assert torch.equal(L.shared, w0)
