"""Host-side logic of the decode driver: the length schedules it hands to the
kernels follow the eviction rule (append, then evict to B once the live
length exceeds B + buffer)."""
from paper_2608_15797_amd.pipeline import base_length_schedule, helper_suffix_schedule
from paper_2608_15797_amd.workloads import WORKLOADS
from oracle.run import BaseOracle


def test_base_schedule_matches_oracle_loop():
    import numpy as np
    S, L, Hkv, Hq, D, B, W, buffer, T = 1, 1, 1, 2, 8, 8, 3, 4, 45
    orc = BaseOracle(S, L, Hkv, Hq, D, B, W, buffer, np.float32, 1.0)
    sched = base_length_schedule(T, B, buffer)
    g = np.random.default_rng(0)
    for t in range(T):
        orc.step(t, g.standard_normal((S, L, Hq, D)).astype(np.float32),
                 g.standard_normal((S, L, Hkv, D)).astype(np.float32),
                 g.standard_normal((S, L, Hkv, D)).astype(np.float32))
        n_after_append = orc.events[-1]["n"] if orc.events and orc.events[-1]["t"] == t else orc.n
        assert sched[t] == n_after_append


def test_workload_eviction_counts():
    """Eviction events per run: tiny 4; 7B B=128 prompt 256 + 1024 steps: 8
    (the cap is 257, so the first eviction is the first decode token); B=64
    workloads evict twice inside their 256-token prompt."""
    def events(wl):
        b = wl.base
        s = base_length_schedule(b.prompt + wl.steps, b.B, b.buffer)
        return [t for t, n in enumerate(s) if n > b.B + b.buffer]
    assert len(events(WORKLOADS["tiny"])) == 4
    e = events(WORKLOADS["base7b"])
    assert len(e) == 8 and e[0] == 256
    e = events(WORKLOADS["base7b_helper"])
    assert e[:2] == [128, 193] and len(e) == 2 + 63
    e = events(WORKLOADS["base72b_helper"])
    assert e[:2] == [128, 193] and len(e) == 2 + 126


def test_helper_schedule_wraps_at_512():
    s = helper_suffix_schedule(1100, 512)
    assert s[0] == 1 and s[511] == 512 and s[512] == 1 and s[1099] == 1099 - 1024 + 1
