"""The stored profile of the benchmark's default command agrees with the
benchmark's own accounting: the roofline of the dominant call (helper
attention) recomputed from the kernel trace's timed-window durations and the
algorithmic bytes of that window's steps, and the traffic record taken over
the same window's dispatches."""
import json
import os
import re

from paper_2608_15797_amd.benchplan import PEAK_HBM_GBPS, Schedule, place_window, step_bytes, window_stats
from paper_2608_15797_amd.workloads import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROF = os.path.join(ROOT, "profiles")


def _timed_window_durations(path):
    """Kernel -> average microseconds in the first block of the trace summary
    (the timed pass)."""
    text = open(path).read()
    block = text.split("```")[1]
    out = {}
    for line in block.strip().splitlines():
        m = re.match(r"duration\s+(.*?)\s+calls\s+(\d+)\s+avg_us\s+([\d.]+)", line)
        out[m.group(1)] = (int(m.group(2)), float(m.group(3)))
    return out


def test_default_roofline_from_stored_profile():
    wl = WORKLOADS["base72b_helper"]
    K, W = 20, 5   # the driver's command
    s0 = place_window(wl, K, W)
    sch = Schedule(wl, s0 + K + 1)
    alg = sum(step_bytes(wl, sch, i)["helper_attn"] for i in range(s0, s0 + K)) / K
    dur = _timed_window_durations(os.path.join(PROF, "base72b_helper_kernel_trace.md"))
    helper = [v for k, v in dur.items() if "attn_prefix_bf16" in k or "attn_cache_bf16<128, true" in k]
    assert len(helper) == 2 and all(n == K for n, _ in helper)
    us = sum(t for _, t in helper)
    frac = alg / (us * 1e-6) / 1e9 / PEAK_HBM_GBPS
    # The benchmark's roofline fraction in the profiled run itself (its HIP
    # events around the same calls), as the profile records it, lies within
    # 1 percent of the one recomputed from the kernel durations.
    text = open(os.path.join(PROF, "base72b_helper_kernel_trace.md")).read()
    bench_frac = float(re.search(r"between its events \((0\.\d+)\)", text).group(1))
    assert abs(frac - bench_frac) / bench_frac < 0.01
    # The traffic record covers the same window: same steps, and algorithmic
    # bytes per dispatch of the helper call equal to the benchmark's.
    rec = json.load(open(os.path.join(PROF, "traffic_base72b_helper.json")))
    assert rec["window"] == window_stats(wl, sch, s0, K)
    h = rec["calls"]["helper_attn"]
    assert h["alg_bytes_per_dispatch"] == int(round(alg))
    assert 1.0 <= h["bytes_per_call"] / h["alg_bytes_per_dispatch"] < 1.01


def test_suffix_fit_recovers_a_planted_line(tmp_path):
    """profsum --suffix-fit on a synthetic kernel trace: suffix dispatches of
    7 + 0.05 u microseconds (u from the workload's schedule), among other
    dispatches and outside the marker window, give back 7 and 0.05."""
    import sqlite3

    from paper_2608_15797_amd import profsum
    wl = WORKLOADS["helper4k"]
    s0, K = 5, 40
    sch = Schedule(wl, s0 + K + 1)
    db = tmp_path / "run_results.db"
    c = sqlite3.connect(db)
    c.execute("create table kernels (dispatch_id integer, name text, start integer, end integer)")
    rows, t, k = [], 0, 0

    def put(name, us):
        nonlocal t, k
        rows.append((k, name, t, t + int(round(us * 1e3))))
        t += int(round(us * 1e3)) + 100
        k += 1

    suffix = "void kvr::(anonymous namespace)::attn_cache_bf16<128, true, 2, 2, true, 0>(kvr::AttnParams)"
    put(suffix, 999.0)  # before the window
    put("at::native::spin_kernel(long)", 1.0)
    for i in range(K):
        put("void kvr::(anonymous namespace)::attn_prefix_rows_bf16<128, 1, 2, 2>(kvr::AttnParams)", 140.0)
        put(suffix, 7.0 + 0.05 * sch.hlen_host[s0 + i])
    put("at::native::spin_kernel(long)", 1.0)
    put(suffix, 999.0)  # after it
    c.executemany("insert into kernels values (?, ?, ?, ?)", rows)
    c.commit()
    c.close()
    line = {"steps": K, "config": {"workload": "helper4k", "window": {"first_step": s0, "steps": K}}}
    bj = tmp_path / "bench.json"
    bj.write_text("log line\n" + json.dumps(line) + "\n")
    out = profsum.suffix_fit(str(db), str(bj))
    m = re.search(r"duration = ([\d.]+) us \+ ([\d.]+) us x u", out[0])
    assert m and abs(float(m.group(1)) - 7.0) < 0.05 and abs(float(m.group(2)) - 0.05) < 1e-4, out
