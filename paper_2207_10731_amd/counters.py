"""Cache and atomic counters of the library's kernels, summarised.

  python -m paper_2207_10731_amd.counters --out profiles/cache_atomics_c2.md DB1 DB2 ...

Each DB is a rocprofv3 result database of one --pmc pass over the same
command (counters differ per pass).  For each kernel named by --kernels
(default: forward_stream_kernel, forward_kernel and reduce_deposit_kernel) it prints the
per-dispatch average of every counter found, and the derived L2 hit rate
and atomic requests per lookup.
"""
from __future__ import annotations

import argparse
import sqlite3
from collections import defaultdict

KERNELS = ("forward_stream_kernel", "forward_kernel", "reduce_deposit_kernel")


def collect(dbs, kernels=KERNELS):
    vals = defaultdict(dict)
    for db in dbs:
        c = sqlite3.connect(db)
        for name, counter, avg in c.execute(
                "select kernel_name, counter_name, avg(value) from counters_collection "
                "group by kernel_name, counter_name"):
            for k in kernels:
                if f"pss::{k}<" in name or f"pss::{k}(" in name:
                    vals[k][counter] = avg
    return vals


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("dbs", nargs="+")
    ap.add_argument("--lookups", type=float, default=1703936.0)
    ap.add_argument("--command", default="")
    ap.add_argument("--out", default=None)
    ap.add_argument("--kernels", default=",".join(KERNELS),
                    help="comma-separated kernel names (without the pss:: prefix)")
    a = ap.parse_args(argv)
    kernels = tuple(k for k in a.kernels.split(",") if k)
    vals = collect(a.dbs, kernels)
    lines = ["| counter (per dispatch) | " + " | ".join(kernels) + " |",
             "|---|" + "---|" * len(kernels)]
    names = sorted({n for k in kernels for n in vals[k]})
    for n in names:
        lines.append(f"| {n} | " + " | ".join(f"{vals[k].get(n, float('nan')):,.0f}" for k in kernels) + " |")
    derived = []
    for k in kernels:
        v = vals[k]
        if "TCC_HIT_sum" in v and "TCC_MISS_sum" in v:
            tot = v["TCC_HIT_sum"] + v["TCC_MISS_sum"]
            derived.append(f"- {k}: L2 hit rate {v['TCC_HIT_sum'] / tot:.3f} of {tot:,.0f} requests")
        for n in ("TCC_EA0_ATOMIC_sum", "TCP_TCC_ATOMIC_WITHOUT_RET_REQ_sum", "TCC_ATOMIC_sum"):
            if n in v and v[n] > 0:
                derived.append(f"- {k}: {n} {v[n] / a.lookups:.3f} per lookup")
    text = "\n".join(lines + [""] + derived) + "\n"
    if a.command:
        text = f"Command: `{a.command}`\n\n" + text
    if a.out:
        with open(a.out, "w") as f:
            f.write(text)
    print(text)


if __name__ == "__main__":
    main()
