"""Benchmark of the PSS hashed-embedding layer on one MI355X.

One step = pss_forward + pss_backward_update (forward gather/pool, backward
deposit, optimizer step) over one batch of synthetic bags, rotating 4
pre-generated index batches and gradient batches resident in HBM.  The
forward is called with PSS_PREPARE_BACKWARD, as a training step can: on the
headline workload its streamed kernel writes the first stage of the
backward's grouping (keys, rows, digit counts) while it reads the batch's
index and offset entries, and the backward finishes the grouping (379.7
against 391.3 us per step without the flag, on one box).  --no-prepare: the
backward groups the batch itself.  --prepare: each step starts with
pss_prepare_backward instead, the whole grouping on a library stream beside
the forward kernel (slower there: it shares the memory system with a
forward that writes at the streamed rate).

Default workload: criteo-tb-shaped one-hot batch (26 tables with log-uniform
cardinalities in [3, 4e7], Zipf(1.1) indices, batch 65536, d = 128, Z = 32,
shared float32 array of 2.5e6 weights = 10 MB, SGD).

Prints one JSON line on stdout; diagnostics go to stderr.
  value          lookups/s over the timed steps (lookup = one (sample, table,
                 index) row: d gathered, pooled, d deposited)
  roofline       the dominant kernel's floor bytes per launch over its
                 average duration (HIP events on the launch stream, around the
                 pss_forward call, which enqueues that one kernel there) vs the
                 peak of the memory level that bounds it; step_* fields give
                 the same for the whole step.  Floor bytes per level: HBM
                 carries the index/offset/row streams and the dense optimizer
                 pass; the array's own level (one XCD's L2, the memory-side
                 cache, or HBM at 64-byte sector granularity) carries each
                 distinct chunk of the batch once per gather and once per
                 read-modify-write.  Peaks: 8 TB/s for HBM (vendor); streaming
                 reads measured at start-up for the caches (no published
                 figure), reported with the random 64-byte gather rates.
                 Events bracket the calls of every --event-every-th timed step
                 only (10 of 100): each event record costs the stream about
                 4 us, which is counted as step time.  On the steps halfway
                 between (10 more) the library has the dispatch of its
                 reduce-and-deposit kernel record events at the kernel's start
                 and end (no commands added to the stream).
  cpu_baseline   the CPU oracle timed on a prefix of the same batch
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

HBM_PEAK_GBS = 8000.0
ROTATE = 4
PMC_FILE = os.path.join(ROOT, "profiles", "pmc_forward_c2.json")
PMC_REDUCE_FILE = os.path.join(ROOT, "profiles", "pmc_reduce_deposit_c2.json")


# Sources each profiled kernel is compiled from (its own file and the shared
# device headers): a counter summary stays valid while these are unchanged.
KERNEL_SOURCES = {
    "forward_kernel": ["pss_forward.hip"],
    "forward_stream_kernel": ["pss_forward.hip"],
    "reduce_deposit_kernel": ["pss_sorted.hip"],
}
SHARED_HEADERS = ["pss_hash.hpp", "pss_kernels.hpp", "pss_keygen.hpp"]  # device code; pss_launch.hpp only declares


def source_digest(kernel: str = "forward_kernel") -> str:
    """sha256 over the HIP sources a kernel is built from."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2207_10731_amd", "csrc")
    h = hashlib.sha256()
    for name in sorted(KERNEL_SOURCES[kernel] + SHARED_HEADERS):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def kernel_counters(workload: str, kernel: str = "forward_kernel"):
    """The committed counter summary of the forward kernel (kernel =
    "forward_kernel") or of the reduce stage ("reduce_deposit_kernel"), or
    None when it was taken on other kernel sources or another workload."""
    path = PMC_FILE if kernel == "forward_kernel" else PMC_REDUCE_FILE
    try:
        with open(path) as f:
            pmc = json.load(f)
    except (OSError, ValueError):
        return None
    if pmc.get("source_sha256") != source_digest(kernel) or pmc.get("workload") != workload:
        return None
    return pmc


def forward_counters(workload: str):
    return kernel_counters(workload, "forward_kernel")


def counted_traffic(workload: str, kernel: str = "forward_kernel"):
    """HBM bytes per launch from the committed counter summary, or None
    when it was taken on other kernel sources or another workload."""
    pmc = kernel_counters(workload, kernel)
    if pmc is None:
        return None
    return pmc["fetch_kib"] * 1024 * pmc["fetch_scale"] + pmc["write_kib"] * 1024 * pmc["write_scale"]


class ReduceTimer:
    """HIP events recorded at the start and end of the library's
    reduce-and-deposit kernel (pss_debug_reduce_events), one pair per timed
    call.  A pair the
    library never recorded (no such kernel on this workload's path) reads
    as None."""

    def __init__(self, n):
        import ctypes
        self._ct = ctypes
        self.hip = ctypes.CDLL("libamdhip64.so")  # the runtime torch already loaded
        self.pairs = []
        for _ in range(n):
            pair = []
            for _ in range(2):
                h = ctypes.c_void_p()
                if self.hip.hipEventCreate(ctypes.byref(h)) != 0:
                    raise RuntimeError("hipEventCreate failed")
                pair.append(h)
            self.pairs.append(pair)

    def elapsed_ms(self, i):
        ms = self._ct.c_float()
        st = self.hip.hipEventElapsedTime(self._ct.byref(ms), self.pairs[i][0], self.pairs[i][1])
        if st != 0:
            # events never recorded: clear the runtime's last error, which
            # the next HIP call (torch's included) would report otherwise
            self.hip.hipGetLastError()
            return None
        return ms.value

    def close(self):
        for pair in self.pairs:
            for h in pair:
                self.hip.hipEventDestroy(h)
        self.pairs = []


def log(*a):
    print(*a, file=sys.stderr, flush=True)


SECTOR = 64  # bytes a random access of a few bytes moves at HBM (one sector)


def array_level(wl):
    """Memory level the shared array lives in: one XCD's L2 (4 MiB), the
    memory-side cache (256 MiB) or HBM."""
    nbytes = wl.M * (2 if wl.weight_dtype == "bf16" else 4)
    if nbytes <= 4 << 20:
        return "l2"
    if nbytes <= 256 << 20:
        return "cache"
    return "hbm"


def optimizer_bytes(wl):
    """Dense optimizer pass over M when one runs (Adagrad or bf16 storage):
    zero-fill G (4 B write) + read G (4) + read/write w + read/write s."""
    if wl.optimizer == "sgd" and wl.weight_dtype == "f32":
        return 0
    wsz = 2 if wl.weight_dtype == "bf16" else 4
    state = 8 if wl.optimizer == "adagrad" else 0
    return wl.M * (4 + 4 + 2 * wsz + state)


def distinct_chunks(wl, pss, hp, idx, off, dev):
    """Distinct chunk bases of a batch, and distinct 64-byte sectors of the
    array those chunks touch, from the library's export of every chunk base
    (identical lookups share a base; on-chip aggregation moves each once)."""
    import torch
    bases = torch.empty((int(hp.num_indices), wl.C), dtype=torch.int32, device=dev)
    pss.pss_debug_addresses(wl.M, wl.Z, wl.d, hp, idx, off, bases)
    b = bases.view(-1).to(torch.int64) & 0xFFFFFFFF
    del bases
    uniq = torch.unique(b)
    sw = 2 if wl.weight_dtype == "bf16" else 4
    first = uniq * sw // SECTOR
    last = (uniq * sw + wl.Z * sw - 1) // SECTOR  # a chunk may straddle a sector boundary
    sectors = torch.unique(torch.cat([first, last])).numel()
    return int(uniq.numel()), int(sectors)


def traffic(wl, B, N, distinct):
    """Floor bytes of one forward and one backward launch at each memory level.

    HBM: indices (8 B each) + offsets (8 B per bag + 1) + pooled rows (4 B per
    element) in each direction, and the dense optimizer pass when one runs.
    Array level: identical lookups read and update the same chunk, so with
    on-chip aggregation the forward must read each distinct chunk of the batch
    once (Z weights) and the backward must read and write each once (Z
    float32 values).  When the array lives in HBM those accesses are random
    and move whole 64-byte sectors: each distinct sector is read by the
    forward and read and written by the backward.
    distinct = (distinct chunk bases, distinct sectors) of the batch.
    Returns {level: (forward bytes, backward bytes)}.
    """
    sw = 2 if wl.weight_dtype == "bf16" else 4
    chunks, sectors = distinct
    stream = 8 * N + 8 * (wl.T * B + 1)
    rows = 4 * B * wl.T * wl.d
    fwd, bwd = stream + rows, stream + rows + optimizer_bytes(wl)
    level = array_level(wl)
    if level == "hbm":
        return {"hbm": (fwd + sectors * SECTOR, bwd + 2 * sectors * SECTOR)}
    return {"hbm": (fwd, bwd), level: (chunks * wl.Z * sw, 2 * chunks * wl.Z * 4)}


def level_peaks(measured):
    """GB/s per level: the vendor's HBM figure; measured streaming reads for
    the caches, which have no published peak."""
    peaks = {"hbm": (HBM_PEAK_GBS, "vendor")}
    if measured:
        peaks["cache"] = (measured["cache_read_gbs"], "measured streaming read")
        peaks["l2"] = (measured["l2_read_gbs"], "measured streaming read")
    return peaks


def cpu_baseline(wl, x, a, b, budget_s=24.0):
    """Times the CPU oracle (forward + gradient + update, float64) on the first
    B' samples of batch 0, B' doubled until one pass takes >= budget/4.  One
    untimed pass on 256 samples comes first: the first call pays one-off
    costs (first touch of fresh arrays, first use of NumPy routines)."""
    import synth
    from oracle import pss_oracle as o
    w = synth.make_weights(wl)
    s = np.zeros(wl.M, dtype=np.float32) if wl.optimizer == "adagrad" else None

    def one_pass(Bp):
        lens = np.diff(x.offsets).reshape(wl.T, x.B)[:, :Bp]
        off = np.zeros(wl.T * Bp + 1, dtype=np.int64)
        np.cumsum(lens.ravel(), out=off[1:])
        starts = x.offsets[:-1].reshape(wl.T, x.B)[:, :Bp]
        idx = np.concatenate([x.indices[st:st + ln] for st, ln in zip(starts.ravel(), lens.ravel())])
        g = np.random.default_rng(7).standard_normal((Bp, wl.T * wl.d), dtype=np.float32)
        t0 = time.perf_counter()
        o.forward64(w, wl.M, wl.Z, wl.d, wl.T, Bp, a, b, idx, off, wl.weight_dtype)
        o.backward_update(w, s, wl.M, wl.Z, wl.d, wl.T, Bp, a, b, idx, off, g, wl.lr, wl.eps,
                          wl.weight_dtype)
        return idx.shape[0], time.perf_counter() - t0

    one_pass(min(256, x.B))
    Bp = 256
    best = None
    spent = 0.0
    while True:
        n, dt = one_pass(min(Bp, x.B))
        spent += dt
        best = (n, dt, min(Bp, x.B))
        if dt >= budget_s / 4 or Bp >= x.B or spent + 2 * dt > budget_s:
            break
        Bp *= 2
    n, dt, Bp = best
    host = os.cpu_count()
    avail = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else host
    return {"value": n / dt, "unit": "lookups/s", "cores": 1, "host_cores": host,
            "available_cores": avail, "kind": "oracle",
            "sample": f"first {Bp} of {x.B} samples of batch 0 ({n} lookups, all {wl.T} tables), "
                      f"one forward+gradient+update pass, float64 NumPy, single thread: "
                      f"1 of {host} host cores ({avail} available to the process)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="c2")
    ap.add_argument("--variant", default="auto", choices=["auto", "atomic", "sorted", "sparse"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--prepare", action="store_true",
                    help="start each step with pss_prepare_backward (the grouping beside the "
                         "forward) instead of the flag on pss_forward")
    ap.add_argument("--no-prepare", action="store_true",
                    help="no preparation: the backward groups the batch itself")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip measuring the L2 / memory-side cache / HBM denominators")
    ap.add_argument("--event-every", type=int, default=10,
                    help="time the calls of every n-th timed step with HIP events")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the layer's multi-GPU "
              f"sharding is a design note, not a measured path", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_2207_10731_amd import pss

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda", 0)
    wl = synth.get(args.config)
    flags = {"auto": pss.PSS_BWD_AUTO, "atomic": pss.PSS_BWD_ATOMIC,
             "sorted": pss.PSS_BWD_SORTED, "sparse": pss.PSS_BWD_SPARSE}[args.variant]
    dt_code = pss.PSS_BF16 if wl.weight_dtype == "bf16" else pss.PSS_F32

    measured = None
    if not args.no_peaks:
        from paper_2207_10731_amd import peaks
        t0 = time.perf_counter()
        measured = peaks.measure(dev)
        log("[bench] measured peaks (GB/s): " + ", ".join(f"{k} {v:.0f}" for k, v in measured.items())
            + f" in {time.perf_counter() - t0:.1f}s")
    t0 = time.perf_counter()
    xs = [synth.make_inputs(wl, batch=k) for k in range(ROTATE)]
    log(f"[bench] {wl.name}: inputs generated in {time.perf_counter() - t0:.1f}s; "
        f"N per batch {[x.N for x in xs]}")
    w = synth.make_weights(wl)
    if wl.weight_dtype == "bf16":
        shared = torch.from_numpy(w.view(np.int16)).to(dev).view(torch.bfloat16)
    else:
        shared = torch.from_numpy(w).to(dev)
    state = torch.zeros(wl.M, dtype=torch.float32, device=dev) if wl.optimizer == "adagrad" else None
    idx = [torch.from_numpy(x.indices).to(dev) for x in xs]
    off = [torch.from_numpy(x.offsets).to(dev) for x in xs]
    gen = torch.Generator(device=dev)
    gen.manual_seed(wl.data_seed)
    grads = [torch.randn((wl.B, wl.T * wl.d), generator=gen, device=dev) for _ in range(ROTATE)]
    out = torch.empty((wl.B, wl.T * wl.d), dtype=torch.float32, device=dev)
    prepare = args.prepare and not args.no_prepare
    in_forward = not args.prepare and not args.no_prepare
    fwd_flags = flags | (pss.PSS_PREPARE_BACKWARD if in_forward else 0)
    hps = [pss.make_hash_params(wl.hash_seed, num_tables=wl.T, batch=wl.B, num_indices=x.N,
                                weight_dtype=dt_code, eps=wl.eps, flags=fwd_flags) for x in xs]
    torch.cuda.synchronize()

    def step(k, ev=None, red=None):
        r = k % ROTATE
        if prepare:
            pss.pss_prepare_backward(wl.M, wl.Z, wl.d, hps[r], idx[r], off[r])
        if ev is not None:
            ev[0].record()
        pss.pss_forward(shared, wl.M, wl.Z, wl.d, hps[r], idx[r], off[r], out)
        if ev is not None:
            ev[1].record()
        if red is not None:
            pss.pss_debug_reduce_events(red[0], red[1])
        pss.pss_backward_update(shared, state, wl.M, wl.Z, wl.d, hps[r], idx[r], off[r], grads[r],
                                wl.lr)
        if red is not None:
            pss.pss_debug_reduce_events()
        if ev is not None:
            ev[2].record()

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    every = max(1, args.event_every)
    evs = {k: [torch.cuda.Event(enable_timing=True) for _ in range(3)]
           for k in range(0, args.steps, every)}
    # the reduce kernel is timed on the steps halfway between the bracketed
    # ones (two more event records per timed call, kept out of the forward
    # and backward brackets)
    red_phase = every // 2 if every > 1 else 0
    red_steps = [k for k in range(args.steps) if k % every == red_phase]
    timer = ReduceTimer(len(red_steps))
    red = {k: timer.pairs[i] for i, k in enumerate(red_steps)}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(k, evs.get(k), red.get(k))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    red_ms = [timer.elapsed_ms(i) for i in range(len(red_steps))]
    timer.close()
    red_ms = np.array(red_ms, dtype=float) if red_ms and all(x is not None for x in red_ms) else None

    fwd_ms = np.array([e[0].elapsed_time(e[1]) for e in evs.values()])
    bwd_ms = np.array([e[1].elapsed_time(e[2]) for e in evs.values()])
    lookups = sum(xs[k % ROTATE].N for k in range(args.steps))
    value = lookups / wall
    ms_per_step = 1e3 * wall / args.steps
    N_avg = lookups / args.steps

    f_avg, b_avg = fwd_ms.mean() * 1e-3, bwd_ms.mean() * 1e-3
    distinct = distinct_chunks(wl, pss, hps[0], idx[0], off[0], dev)
    log(f"[bench] batch 0: {distinct[0]} distinct chunk bases of {xs[0].N * wl.C} chunks, "
        f"{distinct[1]} distinct 64-byte sectors")
    tr = traffic(wl, wl.B, N_avg, distinct)
    peaks_gbs = level_peaks(measured)
    t_step = wall / args.steps
    levels = {}
    for lv, (fb_l, bb_l) in tr.items():
        pk = peaks_gbs.get(lv)
        levels[lv] = {"bytes_per_step": fb_l + bb_l, "forward_bytes": fb_l, "backward_bytes": bb_l,
                      "peak_gbs": None if pk is None else pk[0],
                      "peak_source": None if pk is None else pk[1],
                      "t_star_us": None if pk is None else (fb_l + bb_l) / (pk[0] * 1e9) * 1e6,
                      "achieved_gbs": (fb_l + bb_l) / t_step / 1e9}
    timed = {lv: v for lv, v in levels.items() if v["t_star_us"] is not None}
    step_bound = max(timed, key=lambda lv: timed[lv]["t_star_us"])
    t_star = timed[step_bound]["t_star_us"] * 1e-6
    # Kernels timed live: pss_forward launches exactly one kernel (events
    # around the call time it); the library has the reduce-and-deposit
    # kernel's dispatch record events at its start and end on request.  Each kernel's bound is the level
    # whose floor time is largest for its own bytes; the roofline object
    # describes the longer of the two (the dominant kernel), and both are
    # listed under "kernels".  Kernel names are those the committed counters
    # recorded (pss_forward launches the streamed or the tiled kernel, by the
    # batch's shape).
    fwd_lv = max(timed, key=lambda lv: timed[lv]["forward_bytes"] / peaks_gbs[lv][0])
    pmc = forward_counters(wl.name)
    kernels = {"forward": {
        "kernel": pmc["kernel"].split("(")[0] if pmc is not None else "pss_forward",
        "bound": fwd_lv, "bytes_per_launch": tr[fwd_lv][0], "avg_launch_us": f_avg * 1e6,
        "peak": peaks_gbs[fwd_lv][0], "timed_launches": len(evs),
        "traffic": counted_traffic(wl.name) if fwd_lv == "hbm" else None}}
    if red_ms is not None:
        # the reduce stage reads every lookup's gradient row and its grouped
        # (key, row) pair: HBM-bound
        pmc_r = kernel_counters(wl.name, "reduce_deposit_kernel")
        kernels["reduce"] = {
            "kernel": pmc_r["kernel"].split("(")[0] if pmc_r is not None else "reduce_deposit_kernel",
            "bound": "hbm", "bytes_per_launch": 4.0 * wl.B * wl.T * wl.d + 8.0 * N_avg,
            "avg_launch_us": red_ms.mean() * 1e3, "peak": peaks_gbs["hbm"][0],
            "timed_launches": len(red_ms),
            "traffic": counted_traffic(wl.name, "reduce_deposit_kernel")}
    for kv in kernels.values():
        kv["achieved"] = kv["bytes_per_launch"] / (kv["avg_launch_us"] * 1e-6) / 1e9
        kv["frac"] = kv["achieved"] / kv["peak"]
    dom_key = max(kernels, key=lambda k: kernels[k]["avg_launch_us"])
    dk = kernels[dom_key]
    achieved = kernels["forward"]["achieved"]
    fb, bb = tr["hbm"]
    log(f"[bench] forward   median {np.median(fwd_ms)*1e3:.1f} us  p10 {np.percentile(fwd_ms,10)*1e3:.1f}"
        f"  p90 {np.percentile(fwd_ms,90)*1e3:.1f}  -> {achieved:.0f} GB/s at level {fwd_lv}")
    log(f"[bench] backward  median {np.median(bwd_ms)*1e3:.1f} us  p10 {np.percentile(bwd_ms,10)*1e3:.1f}"
        f"  p90 {np.percentile(bwd_ms,90)*1e3:.1f}  -> {bb/b_avg/1e9:.0f} GB/s (HBM floor bytes)")
    if "reduce" in kernels:
        kr = kernels["reduce"]
        log(f"[bench] reduce    mean {kr['avg_launch_us']:.1f} us  -> {kr['achieved']:.0f} GB/s, "
            f"frac {kr['frac']:.3f} (kernel only)")
    log(f"[bench] dominant kernel: {dom_key} ({dk['kernel']})")
    for lv, v in levels.items():
        tstar = "n/a" if v["t_star_us"] is None else f"{v['t_star_us']:.1f} us"
        log(f"[bench] level {lv}: {v['bytes_per_step']/1e6:.1f} MB/step, peak "
            f"{v['peak_gbs'] if v['peak_gbs'] is None else round(v['peak_gbs'])} GB/s "
            f"({v['peak_source']}), T* {tstar}, achieved {v['achieved_gbs']:.0f} GB/s")
    log(f"[bench] step {ms_per_step*1e3:.1f} us, T* {t_star*1e6:.1f} us ({step_bound}), "
        f"frac {t_star/t_step:.3f}")

    cpu = None
    if not args.no_cpu_baseline:
        from oracle import pss_oracle as o
        a, b = o.hash_params_from_seed(wl.hash_seed)
        t0 = time.perf_counter()
        cpu = cpu_baseline(wl, xs[0], a, b)
        log(f"[bench] cpu baseline {cpu['value']:.3e} lookups/s in {time.perf_counter()-t0:.1f}s")

    rec = {
        "metric": "hashed-embedding lookups/sec (fwd+bwd+update) + achieved GB/s vs roofline",
        "value": value,
        "unit": "lookups/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if wl.weight_dtype == "f32" else "bf16-storage/f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "tables": wl.T, "batch": wl.B, "d": wl.d, "Z": wl.Z,
                   "M": wl.M, "storage": wl.weight_dtype, "optimizer": wl.optimizer,
                   "bags": wl.bag, "indices": wl.index_dist, "variant": args.variant, "prepare_backward": "call" if prepare else ("in forward" if in_forward else False),
                   "lookups_per_step": N_avg},
        "roofline": {"bound": dk["bound"], "kernel": dk["kernel"], "achieved": dk["achieved"],
                     "peak": dk["peak"], "unit": "GB/s", "frac": dk["frac"],
                     "traffic": dk["traffic"],
                     "bytes_per_launch": dk["bytes_per_launch"], "avg_launch_us": dk["avg_launch_us"],
                     "timed_launches": dk["timed_launches"],
                     "kernels": kernels,
                     "step_bound": step_bound, "step_t_star_us": t_star * 1e6,
                     "step_frac": t_star / t_step,
                     "step_hbm_bytes": fb + bb,
                     "levels": levels, "measured_peaks_gbs": measured,
                     "distinct_chunks_batch0": distinct[0], "distinct_sectors_batch0": distinct[1],
                     "forward_us": f_avg * 1e6, "backward_update_us": b_avg * 1e6,
                     "backward_update_hbm_bytes": bb,
                     "backward_update_gbs": bb / b_avg / 1e9},
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
