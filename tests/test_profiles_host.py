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
