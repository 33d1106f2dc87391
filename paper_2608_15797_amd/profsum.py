"""Summarise rocprofv3 result databases as short text.

    python -m paper_2608_15797_amd.profsum [--window A B] DIR [DIR ...]
    python -m paper_2608_15797_amd.profsum --traffic OUT.json --workload NAME \
        --calib-bytes N [--window A B] FETCH_DIR WRITE_DIR

The first form prints, for every *_results.db under each DIR, per kernel the
dispatch count and average duration, and the per-dispatch average of every
collected PMC counter (FETCH_SIZE / WRITE_SIZE in KiB). Kernels whose name
contains "copy" are listed too, tagged "copy <name> grid=<grid size>".

The second form turns one FETCH_SIZE pass and one WRITE_SIZE pass into HBM
bytes per library call: each counter is scaled by the factor that maps its
reading on a plain copy kernel of known size (N bytes read and N bytes
written per dispatch; the copy whose WRITE_SIZE is within 10% of N) onto N,
and the kernels that make up one call (CALL_KERNELS) are summed. Each call's
entry carries a hash of its kernel sources (CALL_SOURCES) so that a reader
can tell whether it was taken on the kernels it runs. Per-dispatch averages
run over every dispatch of the profiled program, so the passes should run
the same steps as the measurement they are compared with.

--window A B restricts both forms to the library dispatches issued between
marker dispatch A and marker dispatch B (0-based, in issue order); the
markers are the one-thread spin kernels (torch.cuda._sleep) that bench.py and
trafficrun launch around each of their passes. The calibration copy is
always taken from the whole run.
"""
from __future__ import annotations

import argparse
import collections
import glob
import hashlib
import json
import os
import re
import sqlite3

CSRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")
# Sources whose kernels each call runs (a record stays valid while they do not change).
CALL_SOURCES = {
    "base_attn": ("attn.hip", "kvr_device.h"),
    "base_attn_entropy": ("attn.hip", "entropy_common.h", "sampler_common.h", "kvr_device.h"),
    "helper_attn": ("attn.hip", "attn_wide.hip", "kvr_device.h"),
    "helper_attn_entropy": ("attn.hip", "attn_wide.hip", "entropy_common.h", "sampler_common.h", "kvr_device.h"),
    "evict": ("evict.hip", "kvr_device.h"),
    "entropy": ("entropy.hip", "entropy_common.h", "kvr_device.h"),
}

# Kernels launched by one call of each hot-path entry point, by call name; a
# pattern starting with "?" names a kernel the call launches only for some
# shapes (the entropy merge, absent when whole rows go to one workgroup).
CALL_KERNELS = {
    # The evicted-cache kernel without entropy rows (last template argument 0)
    # and with them (1: bf16 logits, 2: float32 logits).
    "base_attn": (r"attn_cache_bf16<\d+, false, \d+, \d+, (true|false), 0>",),
    "base_attn_entropy": (r"attn_cache_bf16<\d+, false, \d+, \d+, (true|false), [12]>",),
    "helper_attn": (r"attn_prefix_bf16<", r"attn_cache_bf16<\d+, true"),
    # The context kernel with the logit rows in front, then the suffix kernel.
    "helper_attn_entropy": (r"attn_prefix_rows_bf16<", r"attn_cache_bf16<\d+, true"),
    "evict": (r"evict_topb_kernel",),
    "entropy": (r"entropy_kernel<", r"?entropy_merge"),
}


def source_hash(call: str) -> str:
    """Hash of the kernel sources behind one call (see CALL_SOURCES)."""
    h = hashlib.sha256()
    for f in CALL_SOURCES[call]:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def keep(name: str) -> bool:
    return "kvr" in name or "copy" in name.lower()


def is_marker(name: str) -> bool:
    return "spin_kernel" in name


def _cols(c, view):
    return [x[1] for x in c.execute("pragma table_info(%s)" % view)]


def _pick(cols, *names):
    low = {x.lower(): x for x in cols}
    for n in names:
        if n in low:
            return low[n]
    return None


def dispatch_rows(db: str) -> list[dict]:
    """Every kernel dispatch of a kernel-trace database as {order, name, dur_ns},
    in issue order."""
    c = sqlite3.connect(db)
    for view in ("kernels", "kernel_dispatch", "rocpd_kernel_dispatch"):
        cols = _cols(c, view)
        if cols:
            break
    else:
        raise SystemExit("%s: no kernel dispatch table" % db)
    name = _pick(cols, "name", "kernel_name")
    start, end = _pick(cols, "start", "start_timestamp"), _pick(cols, "end", "end_timestamp")
    order = _pick(cols, "dispatch_id", "correlation_id", "id")
    if not (name and start and end and order):
        raise SystemExit("%s: unexpected columns %s" % (db, cols))
    rows = [dict(order=r[0], name=r[1] or "", dur_ns=float(r[3]) - float(r[2]))
            for r in c.execute('select "%s", "%s", "%s", "%s" from %s' % (order, name, start, end, view))]
    rows.sort(key=lambda r: r["order"])
    return rows


def window_orders(rows: list[dict], window) -> tuple:
    """(first, last) issue order strictly between marker dispatches A and B."""
    if window is None:
        return None
    marks = [r["order"] for r in rows if is_marker(r["name"])]
    a, b = window
    if b >= len(marks):
        raise SystemExit("window %s: only %d markers in the run" % (window, len(marks)))
    return marks[a], marks[b]


def in_window(order, bounds) -> bool:
    return bounds is None or bounds[0] < order < bounds[1]


def window_stats(db: str, window) -> list[str]:
    """Per-kernel dispatch count and average duration within a marker window,
    then the per-dispatch average of every collected PMC counter there."""
    rows = dispatch_rows(db)
    bounds = window_orders(rows, window)
    agg = collections.defaultdict(lambda: [0.0, 0])
    for r in rows:
        if keep(r["name"]) and in_window(r["order"], bounds):
            agg[r["name"]][0] += r["dur_ns"]
            agg[r["name"]][1] += 1
    out = ["duration  %-78s calls %7d  avg_us %10.2f" % (n[:78], k, t / k / 1e3)
           for n, (t, k) in sorted(agg.items(), key=lambda x: -x[1][0])]
    for (name, cn), (v, n) in sorted(counters(db, window).items()):
        out.append("counter   %-78s %-24s avg %16.1f  (dispatches %d)" % (name[:78], cn, v / n, n))
    return out


SUFFIX_KERNEL = re.compile(r"attn_cache_bf16<\d+, true")


def suffix_fit(db: str, bench_json: str, window=(0, 1)) -> list[str]:
    """Least-squares fit of the helper suffix kernel's duration against the
    suffix length u of every step of a bench.py timed pass (the dispatches
    between markers A and B of a kernel trace of that command): duration =
    fixed + per_key * u. per_key against the bytes of one more suffix key
    (K and V rows of every candidate's (layer, KV head) units) is the
    kernel's streaming rate; fixed is what a call costs whatever u is."""
    import numpy as np

    from .benchplan import Schedule
    from .workloads import WORKLOADS
    with open(bench_json) as fh:
        line = json.loads(fh.read().strip().splitlines()[-1])
    wl = WORKLOADS[line["config"]["workload"]]
    h = wl.helper
    s0, K = line["config"]["window"]["first_step"], line["steps"]
    rows = dispatch_rows(db)
    bounds = window_orders(rows, window)
    dur = np.array([r["dur_ns"] / 1e3 for r in rows
                    if SUFFIX_KERNEL.search(r["name"]) and in_window(r["order"], bounds)])
    if len(dur) != K:
        raise SystemExit("%s: %d suffix dispatches in the window, %d timed steps" % (db, len(dur), K))
    sch = Schedule(wl, s0 + K + 1)
    u = np.array([sch.hlen_host[s0 + i] for i in range(K)], dtype=float)
    fixed, per_key = np.linalg.lstsq(np.vstack([np.ones(K), u]).T, dur, rcond=None)[0]
    resid = dur - (fixed + per_key * u)
    key_bytes = h.S * h.L * h.Hkv * 2 * h.D * (4 if wl.dtype == "f32" else 2)
    mean = dur.mean()
    return ["suffix kernel, %s, %d timed steps (u = %d..%d, mean %.1f): duration = %.1f us + %.4f us x u "
            "(rms residual %.1f us)" % (wl.name, K, u.min(), u.max(), u.mean(), fixed, per_key,
                                        float(np.sqrt((resid ** 2).mean()))),
            "  mean call %.1f us, fixed part %.1f%%; one more suffix key moves %d bytes: %.2f TB/s marginal"
            % (mean, 100 * fixed / mean, key_bytes, key_bytes / (per_key * 1e-6) / 1e12)]


def _dbs(d: str) -> list[str]:
    return sorted(glob.glob(d + "/**/*_results.db", recursive=True))


def counters(db: str, window=None) -> dict:
    """{(tag, counter): (sum of values, dispatches)}; copies are tagged by grid.
    With a marker window, library kernels count only inside it (copies always)."""
    c = sqlite3.connect(db)
    cols = [x[1] for x in c.execute("pragma table_info(counters_collection)")]
    agg = collections.defaultdict(lambda: [0.0, 0])
    if not cols:
        return agg
    order = _pick(cols, "dispatch_id", "correlation_id")
    rows = [dict(zip(cols, row)) for row in c.execute("select * from counters_collection")]
    if not rows:  # a kernel trace: the view exists, empty
        return agg
    bounds = None
    if window is not None:
        if order is None:
            raise SystemExit("%s: counters have no dispatch order column (%s)" % (db, cols))
        marks = sorted({r[order] for r in rows if is_marker(r.get("kernel_name") or "")})
        a, b = window
        if b >= len(marks):
            raise SystemExit("window %s: only %d markers in %s" % (window, len(marks), db))
        bounds = (marks[a], marks[b])
    for r in rows:
        name = r.get("kernel_name") or ""
        if not keep(name):
            continue
        if "copy" not in name.lower() and not in_window(r[order] if order else 0, bounds):
            continue
        tag = name
        if "copy" in name.lower():
            tag = "copy %s grid=%s" % (name[:50], r.get("grid_size", r.get("grid_x", "?")))
        a = agg[(tag, r.get("counter_name"))]
        a[0] += float(r.get("value") or 0.0)
        a[1] += 1
    return agg


def summarise(db: str) -> list[str]:
    c = sqlite3.connect(db)
    out = []
    rows = list(c.execute("select name, total_calls, average from top_kernels"))
    for name, calls, avg in rows:
        if keep(name):
            out.append("duration  %-78s calls %7d  avg_us %10.2f" % (name[:78], calls, avg))
    for (name, cn), (v, n) in sorted(counters(db).items()):
        out.append("counter   %-78s %-24s avg %16.1f  (dispatches %d)" % (name[:78], cn, v / n, n))
    return out


def _per_dispatch(dirs: list[str], counter: str, window=None) -> dict:
    per = {}
    for d in dirs:
        for db in _dbs(d):
            for (tag, cn), (v, n) in counters(db, window).items():
                if cn == counter:
                    per[tag] = (v / n, n)
    return per


def traffic(fetch_dir: str, write_dir: str, calib_bytes: int, workload: str, window=None) -> dict:
    fetch = _per_dispatch([fetch_dir], "FETCH_SIZE", window)
    write = _per_dispatch([write_dir], "WRITE_SIZE", window)
    kib = calib_bytes / 1024.0
    cal = [t for t in write if t.startswith("copy ") and abs(write[t][0] - kib) <= 0.1 * kib]
    if len(cal) != 1 or cal[0] not in fetch:
        raise SystemExit("no unique calibration copy of %d bytes among %s" % (calib_bytes, sorted(write)))
    tag = cal[0]
    f_read = calib_bytes / (fetch[tag][0] * 1024.0)
    f_write = calib_bytes / (write[tag][0] * 1024.0)
    calls = {}
    for call, pats in CALL_KERNELS.items():
        parts, rd, wr = [], 0.0, 0.0
        for p in pats:
            optional = p.startswith("?")
            ks = [k for k in fetch if re.search(p.lstrip("?"), k) and k in write]
            if optional and not ks:
                continue
            if len(ks) != 1:
                break
            k = ks[0]
            parts.append(dict(kernel=k, dispatches=fetch[k][1],
                              read_bytes=int(fetch[k][0] * 1024 * f_read),
                              write_bytes=int(write[k][0] * 1024 * f_write)))
            rd += parts[-1]["read_bytes"]
            wr += parts[-1]["write_bytes"]
        else:
            calls[call] = dict(read_bytes=int(rd), write_bytes=int(wr), bytes_per_call=int(rd + wr),
                               source_hash=source_hash(call), kernels=parts)
    return dict(workload=workload,
                calibration=dict(kernel=tag, bytes=calib_bytes, fetch_factor=round(f_read, 4),
                                 write_factor=round(f_write, 4)),
                calls=calls)


def attach_alg(rec: dict, log_path: str) -> None:
    """Add the profiled program's algorithmic bytes per dispatch (the last
    JSON line of its output holding "alg_bytes_per_dispatch") to each call of
    a traffic record, with the measured/algorithmic ratio; the dispatch
    counts of the two must agree. The line's "window" (the decode steps it
    covers) is copied to the record."""
    alg = None
    with open(log_path) as fh:
        for line in fh:
            line = line.strip()
            if line.startswith("{") and "alg_bytes_per_dispatch" in line:
                alg = json.loads(line)
    if alg is None:
        raise SystemExit("no algorithmic-bytes line in %s" % log_path)
    for call, c in rec["calls"].items():
        if call not in alg["alg_bytes_per_dispatch"]:
            continue
        n = alg["dispatches"][call]
        got = {k["dispatches"] for k in c["kernels"]}
        if got != {n}:
            raise SystemExit("%s: %s dispatches counted, %d run" % (call, sorted(got), n))
        c["alg_bytes_per_dispatch"] = alg["alg_bytes_per_dispatch"][call]
        c["measured_over_alg"] = round(c["bytes_per_call"] / c["alg_bytes_per_dispatch"], 4)
    if "window" in alg:
        rec["window"] = alg["window"]


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("dirs", nargs="+")
    ap.add_argument("--traffic", help="write the per-call traffic record to this JSON file")
    ap.add_argument("--workload", default="")
    ap.add_argument("--calib-bytes", type=int, default=1 << 30)
    ap.add_argument("--alg", help="output of the profiled program: add its algorithmic bytes per dispatch")
    ap.add_argument("--window", nargs=2, type=int, metavar=("A", "B"),
                    help="only the dispatches between marker dispatches A and B")
    ap.add_argument("--suffix-fit", metavar="BENCH_JSON",
                    help="fit the helper suffix kernel's duration against the suffix length over the timed "
                         "pass of this bench.py output (one trace directory; --window defaults to 0 1)")
    args = ap.parse_args(argv)
    window = tuple(args.window) if args.window else None
    if args.suffix_fit:
        if len(args.dirs) != 1:
            raise SystemExit("--suffix-fit takes one kernel-trace result directory")
        for db in _dbs(args.dirs[0]):
            for line in suffix_fit(db, args.suffix_fit, window or (0, 1)):
                print(line)
        return
    if args.traffic:
        if len(args.dirs) != 2:
            raise SystemExit("--traffic takes the FETCH_SIZE and the WRITE_SIZE result directories")
        rec = traffic(args.dirs[0], args.dirs[1], args.calib_bytes, args.workload, window)
        if window is not None:
            rec["marker_window"] = list(window)
        if args.alg:
            attach_alg(rec, args.alg)
        with open(args.traffic, "w") as fh:
            json.dump(rec, fh, indent=1)
        print(json.dumps(rec, indent=1))
        return
    for d in args.dirs:
        for db in _dbs(d):
            print("##", db, "" if window is None else "(marker window %d-%d)" % window)
            for line in (summarise(db) if window is None else window_stats(db, window)):
                print(line)


if __name__ == "__main__":
    main()
