"""Host side of bench.py: the single-GPU guard, the placement of the timed
window and the per-step byte accounting it divides by the measured
durations."""
import os
import subprocess
import sys
from types import SimpleNamespace

import pytest

from paper_2608_15797_amd.pipeline import base_length_schedule, helper_suffix_schedule
from paper_2608_15797_amd.workloads import WORKLOADS

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr
    assert r.stdout == ""


def _decoder_stub(wl):
    b, h = wl.base, wl.helper
    T_prompt = b.prompt if b else 0
    return SimpleNamespace(
        T_prompt=T_prompt,
        blen_host=base_length_schedule(T_prompt + wl.steps, b.B, b.buffer) if b else None,
        hlen_host=helper_suffix_schedule(wl.steps, h.scap) if h else None)


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("name", ["base7b_helper", "base7b", "base72b_helper", "helper4k"])
def test_step_bytes_calls(name, fused):
    from paper_2608_15797_amd import benchplan as bench
    wl = WORKLOADS[name]
    dec = _decoder_stub(wl)
    dec.fuse_entropy = fused
    e = 2  # bf16 logits
    logit_bytes = sum(ls.R * ls.V * e + ls.R * 4 for ls in wl.logits)
    evict_steps = 0
    for i in range(wl.steps):
        out = bench.step_bytes(wl, dec, i)
        if fused and wl.base:
            # The entropies ride in the base-attention launch: that call carries the logit bytes.
            n = dec.blen_host[dec.T_prompt + i]
            assert "entropy" not in out and "base_attn" not in out
            assert out["base_attn_entropy"] == bench.acc.base_attn_bytes(wl, n) + logit_bytes
            assert ("helper_attn" in out) == (wl.helper is not None)
        elif fused:
            # Helper only: they ride in the helper's context launch.
            assert "entropy" not in out and "helper_attn" not in out
            assert out["helper_attn_entropy"] == bench.acc.helper_attn_bytes(wl, dec.hlen_host[i]) + logit_bytes
        else:
            # One batched entropy call per step covers every logit set.
            assert out["entropy"] == logit_bytes
            assert ("base_attn" in out) == (wl.base is not None)
            assert ("helper_attn" in out) == (wl.helper is not None)
        if wl.base:
            n = dec.blen_host[dec.T_prompt + i]
            assert ("evict" in out) == (n > wl.base.B + wl.base.buffer)
            evict_steps += "evict" in out
            # Moved rows never exceed the all-B upper bound.
            if "evict" in out:
                assert bench.step_bytes(wl, dec, i, moved_rows=wl.base.B / 2)["evict"] < out["evict"]
    if name == "base7b_helper":
        # B = 64, buffer = 64: one eviction every 65 tokens after the prompt.
        assert evict_steps == 63
        # The default workload's two logit sets: 77.8 MB per step.
        assert logit_bytes == 128 * 152064 * 2 + 128 * 151936 * 2 + 2 * 128 * 4


@pytest.mark.parametrize("name", ["base72b_helper", "base7b_helper", "base7b", "helper4k"])
@pytest.mark.parametrize("K,W", [(20, 5), (1, 0), (33, 5), (100, 32), (0, 32)])
def test_window_placement(name, K, W):
    """The timed window holds an eviction preceded by min(W_policy - 1, K - 1)
    score-streaming steps (with the eviction step, the observation window),
    starts after its warmup, and a default window
    (K = 0: one whole cycle) covers every base length of the eviction cycle
    equally and the helper suffix cycle."""
    from paper_2608_15797_amd.benchplan import Schedule, cycle_steps, place_window, window_stats
    wl = WORKLOADS[name]
    C = cycle_steps(wl)
    K = K or C
    s0 = place_window(wl, K, W)
    assert s0 >= W
    sch = Schedule(wl, s0 + K + 1)
    st = window_stats(wl, sch, s0, K)
    b, h = wl.base, wl.helper
    if b:
        ev = [i for i in range(s0, s0 + K) if sch.evicts(i)]
        assert ev, "no eviction in the window"
        lead = min(b.W - 1, K - 1)
        assert ev[0] - s0 == lead
        assert all(sch.scores(i) for i in range(ev[0] - lead, ev[0] + 1))
        assert st["evictions_in_window"] == len(ev)
    if K == C:
        if b:
            # Whole eviction periods: every live length of the cycle equally often.
            ns = sorted(sch.base_n(i) for i in range(s0, s0 + K))
            per = b.buffer + 1
            assert ns == sorted(list(range(b.B + 1, b.B + b.buffer + 2)) * (K // per))
            assert st["mean_base_len"] == pytest.approx(b.B + (b.buffer + 2) / 2)
        if h:
            assert set(sch.hlen_host[s0:s0 + K]) == set(range(1, h.scap + 1))
    if h and K >= 20:
        assert abs(st["mean_helper_suffix"] - (h.scap + 1) / 2) < 0.1 * h.scap


def test_driver_window_on_the_72b_workload():
    """The driver's --steps 20 --warmup 5 on the default workload: one
    eviction at the last step, all 20 steps streaming window scores."""
    from paper_2608_15797_amd.benchplan import Schedule, place_window, window_stats
    wl = WORKLOADS["base72b_helper"]
    s0 = place_window(wl, 20, 5)
    st = window_stats(wl, Schedule(wl, s0 + 21), s0, 20)
    assert st["evictions_in_window"] == 1 and st["score_steps_in_window"] == 20
    assert abs(st["mean_helper_suffix"] - 256.5) < 5
