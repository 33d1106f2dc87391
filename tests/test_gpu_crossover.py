"""The crossover measurement runs end to end on small shapes of the 7B model
(every route it times goes through the library's kernels) and its report is
self-consistent."""
import math

import pytest

from gpu_util import say

pytestmark = pytest.mark.gpu


def test_crossover_measure_small():
    from paper_2608_15797_amd.crossover import measure
    say("crossover: S=2 B=64 W=16 buffer=16")
    r = measure(S=2, B=64, W=16, buffer=16, lengths=(128, 256, 512))
    assert r["shape"]["B_prime"] == 80
    parts = r["parts_ms"]
    for k, v in parts.items():
        assert math.isfinite(v) and v > 0, k
    for k, v in r["full_ms"].items():
        assert v["context_path"] > 0 and v["cache_kernel"] > 0, k
    a, b = r["fit"]["intercept_ms"], r["fit"]["ms_per_token"]
    step = r["evicted_every_step"]
    assert step["ms"] == pytest.approx(parts["scored_step"] + parts["eviction"], abs=2e-5)
    assert step["ell_star"] == pytest.approx((step["ms"] - a) / b, rel=1e-3, abs=0.2)
    red = r["evicted_every_step_redundancy"]
    assert red["ms"] > step["ms"]
    assert set(step["speedup"]) == {"128", "256", "512"}
