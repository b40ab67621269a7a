"""Writes c1_oracle_slice.json: a slice of the oracle's results on the tiny
workload (4 tables x 1000 rows, d = 16, Z = 4, M = 4096, batch 256, SGD lr 0.1).

Calls only the CPU oracle and the seeded input generator.  Float32 values are
stored as their bit patterns so the fixture is exact.
Run from the repository root:  python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import synth  # noqa: E402
from oracle import pss_oracle as o  # noqa: E402


def main():
    wl = synth.get("c1")
    x = synth.make_inputs(wl)
    w = synth.make_weights(wl)
    g = synth.make_grad(wl)
    a, b = o.hash_params_from_seed(wl.hash_seed)
    bases = o.chunk_bases(wl.M, wl.Z, wl.d, wl.T, x.B, a, b, x.indices, x.offsets)
    out = o.forward(w, wl.M, wl.Z, wl.d, wl.T, x.B, a, b, x.indices, x.offsets)
    w_new, _, G, A, cnt = o.backward_update(w, None, wl.M, wl.Z, wl.d, wl.T, x.B, a, b,
                                            x.indices, x.offsets, g, wl.lr)
    rows = [0, 1, 100, 255]
    elems = [0, 1, 2, 3, 714, 1000, 2047, 4095]
    fixture = {
        "source": "oracle.pss_oracle on synth workload c1 (written by tests/golden/make_golden.py)",
        "a": a, "b": b,
        "bases_first_items": bases[:8].astype(int).tolist(),
        "out_rows": rows,
        "out_bits": [out[r].view(np.uint32).astype(int).tolist() for r in rows],
        "w_new_elems": elems,
        "w_new_bits": w_new[elems].view(np.uint32).astype(int).tolist(),
        "count_elems": cnt[elems].astype(int).tolist(),
    }
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c1_oracle_slice.json")
    with open(path, "w") as f:
        json.dump(fixture, f, indent=1)
        f.write("\n")


if __name__ == "__main__":
    main()
