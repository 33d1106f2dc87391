"""Summarise rocprofv3 result databases as short text.

    python -m paper_2608_15797_amd.profsum DIR [DIR ...]

For every *_results.db under each DIR prints, per kernel, the dispatch count
and average duration, and the per-dispatch average of every collected PMC
counter (FETCH_SIZE / WRITE_SIZE in KiB). Kernels whose name contains "copy"
are listed too: a plain copy of known size is the reference that scales the
byte counters.
"""
from __future__ import annotations

import collections
import glob
import sqlite3
import sys


def keep(name: str) -> bool:
    return "kvr" in name or "copy" in name.lower()


def summarise(db: str) -> list[str]:
    c = sqlite3.connect(db)
    out = []
    rows = list(c.execute("select name, total_calls, average from top_kernels"))
    for name, calls, avg in rows:
        if keep(name):
            out.append("duration  %-78s calls %7d  avg_us %10.2f" % (name[:78], calls, avg))
    cols = [x[1] for x in c.execute("pragma table_info(counters_collection)")]
    if cols:
        # Copies are told apart by grid size (the calibration copy has its own).
        agg = collections.defaultdict(lambda: [0.0, 0])
        for row in c.execute("select * from counters_collection"):
            r = dict(zip(cols, row))
            name = r.get("kernel_name") or ""
            if not keep(name):
                continue
            tag = name[:70]
            if "copy" in name.lower():
                tag = "%s grid=%s" % (name[:50], r.get("grid_size", r.get("grid_x", "?")))
            a = agg[(tag, r.get("counter_name"))]
            a[0] += float(r.get("value") or 0.0)
            a[1] += 1
        for (name, cn), (v, n) in sorted(agg.items()):
            out.append("counter   %-78s %-24s avg %16.1f  (dispatches %d)" % (name, cn, v / n, n))
    return out


def main(argv):
    for d in argv:
        for db in sorted(glob.glob(d + "/**/*_results.db", recursive=True)):
            print("##", db)
            for line in summarise(db):
                print(line)


if __name__ == "__main__":
    main(sys.argv[1:])
