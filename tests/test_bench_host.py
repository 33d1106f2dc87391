"""Host side of bench.py: the single-GPU guard and the per-step byte
accounting it divides by the measured durations."""
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


@pytest.mark.parametrize("name", ["base7b_helper", "base7b", "base72b_helper", "helper4k"])
def test_step_bytes_calls(name):
    import bench
    wl = WORKLOADS[name]
    dec = _decoder_stub(wl)
    e = 2  # bf16 logits
    logit_bytes = sum(ls.R * ls.V * e + ls.R * 4 for ls in wl.logits)
    evict_steps = 0
    for i in range(wl.steps):
        out = bench.step_bytes(wl, dec, i)
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
