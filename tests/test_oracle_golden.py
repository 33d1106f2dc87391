"""The stored tiny-workload seed still qualifies: the oracle reproduces the
recorded eviction tokens and kept positions, and every eviction's candidate
scores are pairwise at least 1e-3 apart (the separation that makes bit-exact
kept-set comparison meaningful)."""
import json
import os

import numpy as np

from oracle.run import min_pairwise_gap
from paper_2608_15797_amd.workloads import WORKLOADS

HERE = os.path.dirname(os.path.abspath(__file__))


def test_tiny_seed_golden():
    import importlib.util
    spec = importlib.util.spec_from_file_location("mg", os.path.join(HERE, "golden", "make_golden.py"))
    mg = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mg)
    g = json.load(open(os.path.join(HERE, "golden", "tiny_seed.json")))
    wl = WORKLOADS["tiny"].with_(seed=g["seed"])
    orc = mg.run_tiny(wl)
    assert [e["t"] for e in orc.events] == g["eviction_tokens"]
    for e, kp in zip(orc.events, g["kept_pos"]):
        assert e["kept_pos"].reshape(-1).tolist() == kp
        assert min_pairwise_gap(e["score"][0, 0, 0], e["n"], wl.base.W) >= 1e-3
        np.testing.assert_allclose(e["score"].sum(), wl.base.W * wl.base.G, rtol=1e-12)
