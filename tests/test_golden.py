"""Stored fixtures under tests/golden/ reproduced by the CPU oracle (no GPU)."""
import json
import os

import numpy as np

import synth
from oracle import brute, pss_oracle as o

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_hand_worked_hash_cases():
    with open(os.path.join(GOLDEN, "hash_cases.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        got = o.bases_for(c["M"], 1, c["C"], c["T"], c["a"], c["b"], np.array([c["i"]]),
                          np.array([c["t"]]))[0, c["j"]]
        assert int(got) == c["base"], c["work"]
        assert brute.base(c["a"], c["b"], c["M"], c["T"], c["C"], c["t"], c["i"], c["j"]) == c["base"]


def test_c1_slice_reproduced():
    with open(os.path.join(GOLDEN, "c1_oracle_slice.json")) as f:
        fx = json.load(f)
    wl = synth.get("c1")
    x = synth.make_inputs(wl)
    w = synth.make_weights(wl)
    g = synth.make_grad(wl)
    a, b = o.hash_params_from_seed(wl.hash_seed)
    assert (a, b) == (fx["a"], fx["b"])
    bases = o.chunk_bases(wl.M, wl.Z, wl.d, wl.T, x.B, a, b, x.indices, x.offsets)
    assert bases[:8].astype(int).tolist() == fx["bases_first_items"]
    out = o.forward(w, wl.M, wl.Z, wl.d, wl.T, x.B, a, b, x.indices, x.offsets)
    for r, bits in zip(fx["out_rows"], fx["out_bits"]):
        assert out[r].view(np.uint32).astype(int).tolist() == bits
    w_new, _, _, _, cnt = o.backward_update(w, None, wl.M, wl.Z, wl.d, wl.T, x.B, a, b,
                                            x.indices, x.offsets, g, wl.lr)
    e = fx["w_new_elems"]
    assert w_new[e].view(np.uint32).astype(int).tolist() == fx["w_new_bits"]
    assert cnt[e].astype(int).tolist() == fx["count_elems"]
