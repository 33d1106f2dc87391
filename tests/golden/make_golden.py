"""Writes tests/golden/tiny_seed.json using only the oracle and the seeded
input generators.

The tiny workload (1 sequence, 1 layer, GQA 4:1, head_dim 64, fp32, B=16,
window 8, buffer 16, prompt 32 + 64 decode steps) is compared with the GPU
bit for bit on its kept sets. That needs inputs whose candidate scores are
pairwise at least 1e-3 apart at every eviction, so near-ties cannot flip a
selection between fp32 (GPU) and fp64 (oracle) arithmetic. This script tries
seeds seed_k = base_seed + 1000 k for k = 0, 1, ... and records the first one
that qualifies, with the gaps and the kept positions the oracle found.

Run: python tests/golden/make_golden.py
"""
import json
import math
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle.run import BaseOracle, min_pairwise_gap  # noqa: E402
from paper_2608_15797_amd import synth  # noqa: E402
from paper_2608_15797_amd.workloads import WORKLOADS  # noqa: E402

SEP = 1e-3


def run_tiny(wl):
    b = wl.base
    orc = BaseOracle(b.S, b.L, b.Hkv, b.Hq, b.D, b.B, b.W, b.buffer, np.float32,
                     1.0 / math.sqrt(b.D))
    for t in range(b.prompt + wl.steps):
        q, k, v = synth.base_token(wl, t)
        orc.step(t, q.numpy(), k.numpy(), v.numpy())
    return orc


def main():
    wl0 = WORKLOADS["tiny"]
    b = wl0.base
    for k in range(1000):
        wl = wl0.with_(seed=wl0.seed + 1000 * k)
        orc = run_tiny(wl)
        gaps = [min(min_pairwise_gap(e["score"][s, l, h], e["n"], b.W)
                    for s in range(b.S) for l in range(b.L) for h in range(b.Hkv))
                for e in orc.events]
        if min(gaps) >= SEP:
            out = dict(workload="tiny", seed=wl.seed, k=k, separation=SEP,
                       min_gaps=gaps, eviction_tokens=[e["t"] for e in orc.events],
                       kept_pos=[e["kept_pos"].reshape(-1).tolist() for e in orc.events])
            path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_seed.json")
            with open(path, "w") as f:
                json.dump(out, f, indent=1)
            print("seed", wl.seed, "k", k, "gaps", gaps)
            return
    raise SystemExit("no qualifying seed in 1000 tries")


if __name__ == "__main__":
    main()
