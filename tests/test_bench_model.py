"""CPU checks of bench.py's roofline model: the floor bytes per launch and
memory level, the dense optimizer pass, which level holds each workload's
array, the peaks, and that the committed counter summary of the dominant
kernel was taken on the present sources (bench.py reports `traffic` only
then)."""
import json
import os

import pytest

import bench
import synth

GB = 1e9


def test_headline_floor_bytes_by_hand():
    """One-hot criteo-tb shape: 8 B per index, 8 B per offset (T*B + 1 of
    them) and 4 B per pooled element, each way; SGD on float32 adds no pass."""
    wl = synth.get("c2")
    N = wl.T * wl.B
    fwd, bwd = bench.traffic(wl, wl.B, N, (529_664, 156_157))["hbm"]
    assert fwd == 8 * N + 8 * (wl.T * wl.B + 1) + 4 * wl.B * wl.T * wl.d == 899_678_216
    assert bwd == fwd
    assert bench.optimizer_bytes(wl) == 0


def test_array_levels():
    assert bench.array_level(synth.get("c1")) == "l2"      # 16 KiB
    assert bench.array_level(synth.get("c2")) == "cache"   # 10 MB
    assert bench.array_level(synth.get("c3")) == "cache"   # 64 MB
    assert bench.array_level(synth.get("c4")) == "hbm"     # 4 GB
    assert bench.array_level(synth.get("c5")) == "cache"   # 128 MB of bfloat16


def test_cache_level_counts_distinct_chunks():
    wl = synth.get("c2")
    levels = bench.traffic(wl, wl.B, wl.T * wl.B, (1000, 10))
    # forward reads each distinct chunk once; the backward reads and writes it
    assert levels["cache"] == (1000 * wl.Z * 4, 2 * 1000 * wl.Z * 4)


def test_hbm_array_counts_sectors():
    wl = synth.get("c4")
    N = wl.T * wl.B
    levels = bench.traffic(wl, wl.B, N, (5, 7))
    stream = 8 * N + 8 * (wl.T * wl.B + 1) + 4 * wl.B * wl.T * wl.d
    assert levels == {"hbm": (stream + 7 * 64, stream + 2 * 7 * 64)}


@pytest.mark.parametrize("key,per_element", [("c3", 4 + 4 + 8 + 8), ("c5", 4 + 4 + 4 + 8)])
def test_optimizer_pass_bytes(key, per_element):
    """G zero-fill and read (4 + 4), the weight read and written (float32 8,
    bfloat16 4), the Adagrad state read and written (8)."""
    wl = synth.get(key)
    assert bench.optimizer_bytes(wl) == wl.M * per_element


def test_peaks():
    assert bench.level_peaks(None) == {"hbm": (8000.0, "vendor")}
    p = bench.level_peaks({"cache_read_gbs": 6000.0, "l2_read_gbs": 20000.0})
    assert p["cache"] == (6000.0, "measured streaming read")
    assert p["l2"] == (20000.0, "measured streaming read")


def test_committed_counters_match_sources():
    """profiles/pmc_*_c2.json carry the sha256 of the sources their kernel
    was built from; both must match the present tree."""
    for kernel, name in (("forward_stream_kernel", "pmc_forward_c2.json"),
                         ("reduce_deposit_kernel", "pmc_reduce_deposit_c2.json")):
        with open(os.path.join(bench.ROOT, "profiles", name)) as f:
            pmc = json.load(f)
        assert pmc["source_sha256"] == bench.source_digest(kernel), name
        assert pmc["workload"] == synth.get("c2").name
        assert f"pss::{kernel}<" in pmc["kernel"], name
    t = bench.counted_traffic(synth.get("c2").name)
    assert t is not None and 0.9 * GB < t < 1.3 * GB
