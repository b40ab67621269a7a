"""Summaries of rocprofv3 result databases (SQLite, rocprofv3 >= 1.0 layout).

  python -m paper_2207_10731_amd.profsum kernels RUN_results.db
      per-kernel dispatch count, average / total duration and share (markdown)

  python -m paper_2207_10731_amd.profsum pmc --workload NAME --kernel SUBSTR \\
      --fetch F.db --write W.db --copy-fetch CF.db --copy-write CW.db \\
      --copy-bytes BYTES --out profiles/pmc_<kernel>_<workload>.json
      FETCH_SIZE / WRITE_SIZE (KiB per dispatch) of the kernel whose name
      contains SUBSTR (forward_stream_kernel, forward_kernel or
      reduce_deposit_kernel), with scale
      factors from a copy kernel that moved BYTES each way, and the sha256 of
      the sources that kernel is built from
"""
from __future__ import annotations

import argparse
import json
import os
import sqlite3
import sys


def kernel_rows(db):
    c = sqlite3.connect(db)
    return c.execute("select name, count(*), avg(duration), sum(duration) from kernels "
                     "group by name order by sum(duration) desc").fetchall()


def counter_avg(db, counter, kernel_substr):
    c = sqlite3.connect(db)
    rows = c.execute("select kernel_name, avg(value), count(value) from counters_collection "
                     "where counter_name = ? group by kernel_name", (counter,)).fetchall()
    hits = [(k, v, n) for k, v, n in rows if kernel_substr in k]
    if len(hits) != 1:
        raise SystemExit(f"{db}: {len(hits)} kernels match {kernel_substr!r} for {counter}")
    return hits[0]


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    k = sub.add_parser("kernels")
    k.add_argument("db")
    p = sub.add_parser("pmc")
    for name in ("workload", "kernel", "fetch", "write", "copy_fetch", "copy_write", "out"):
        p.add_argument("--" + name.replace("_", "-"), required=True)
    p.add_argument("--copy-bytes", type=float, required=True)
    p.add_argument("--command", default="")
    a = ap.parse_args(argv)
    if a.cmd == "kernels":
        rows = kernel_rows(a.db)
        total = sum(r[3] for r in rows)
        print("| kernel | calls | avg us | total us | share |")
        print("|---|---|---|---|---|")
        for name, n, avg, tot in rows:
            print(f"| `{name[:100]}` | {n} | {avg / 1e3:.1f} | {tot / 1e3:.1f} | {100 * tot / total:.1f}% |")
        return
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import bench
    kname, fetch, nf = counter_avg(a.fetch, "FETCH_SIZE", a.kernel)
    _, write, nw = counter_avg(a.write, "WRITE_SIZE", a.kernel)
    _, cfetch, _ = counter_avg(a.copy_fetch, "FETCH_SIZE", "copy_kernel")
    _, cwrite, _ = counter_avg(a.copy_write, "WRITE_SIZE", "copy_kernel")
    rec = {
        "workload": a.workload,
        "kernel": kname,
        "fetch_kib": fetch,
        "write_kib": write,
        "dispatches": [nf, nw],
        "fetch_scale": a.copy_bytes / (cfetch * 1024),
        "write_scale": a.copy_bytes / (cwrite * 1024),
        "copy_fetch_kib": cfetch,
        "copy_write_kib": cwrite,
        "copy_bytes": a.copy_bytes,
        "source_sha256": bench.source_digest(a.kernel),
        "source_files": sorted(bench.KERNEL_SOURCES[a.kernel] + bench.SHARED_HEADERS),
        "command": a.command,
    }
    rec["hbm_bytes_per_dispatch"] = (rec["fetch_kib"] * 1024 * rec["fetch_scale"]
                                     + rec["write_kib"] * 1024 * rec["write_scale"])
    with open(a.out, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(json.dumps(rec, indent=1))


if __name__ == "__main__":
    main()
