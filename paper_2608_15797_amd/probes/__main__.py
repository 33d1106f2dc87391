"""Command line of the measurement probes (see the package docstring)."""
from __future__ import annotations

import argparse
import math
import os
import subprocess
import sys

from . import BIN, build


def entropy_marginal(rows):
    import torch

    from .. import kvr, synth
    dt = torch.bfloat16
    D, V = 128, 152064
    shapes = {"72B (32 x 80 x 8 heads, B=64)": dict(S=32, L=80, Hq=64, Hkv=8, B=64, W=32, buf=64),
              "7B B=128 (64 x 28 x 4 heads)": dict(S=64, L=28, Hq=28, Hkv=4, B=128, W=32, buf=128)}
    logits = synth.normal((max(rows), V), 3.0, 3, "probe", "lg", device="cuda", dtype=dt)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for name, sh in shapes.items():
        S, L, Hq, Hkv, B, W, buf = (sh[k] for k in ("S", "L", "Hq", "Hkv", "B", "W", "buf"))
        cap = (B + buf + 1 + 15) // 16 * 16
        cache = kvr.Cache.empty(S, L, Hkv, cap, D, dt)
        synth.fill_normal_(cache.k, 1.0, 3, "probe", "k")
        synth.fill_normal_(cache.v, 1.0, 3, "probe", "v")
        q = synth.normal((S, L, Hq, D), 1.0, 3, "probe", "q", device="cuda", dtype=dt)
        kn = synth.normal((S, L, Hkv, D), 1.0, 3, "probe", "kn", device="cuda", dtype=dt)
        vn = synth.normal((S, L, Hkv, D), 1.0, 3, "probe", "vn", device="cuda", dtype=dt)
        npos = torch.zeros((S,), dtype=torch.int32, device="cuda")
        scores = torch.zeros((S, L, Hkv, cap), device="cuda")
        out = torch.empty((S, L, Hq, D), dtype=dt, device="cuda")
        pol = kvr.Policy(B, W, buf)
        for n in (B + (buf + 2) // 2, B + buf + 1):
            ln = torch.full((S,), n, dtype=torch.int32, device="cuda")
            H = torch.empty(max(rows), device="cuda")

            def call(R):
                if R:
                    kvr.decode_attn_entropy(cache, ln, q, out, 1 / math.sqrt(D), [kvr.LogitSet(logits[:R], H[:R], V)],
                                            k_new=kn, v_new=vn, new_pos=npos, policy=pol, scores=scores)
                else:
                    kvr.decode_attn(cache, ln, q, out, 1 / math.sqrt(D), k_new=kn, v_new=vn, new_pos=npos,
                                    policy=pol, scores=scores)

            res = {}
            for rep in range(3):  # interleaved passes over every row count
                for R in rows:
                    for _ in range(3):
                        call(R)
                    torch.cuda.synchronize()
                    e0.record()
                    for _ in range(20):
                        call(R)
                    e1.record()
                    torch.cuda.synchronize()
                    res.setdefault(R, []).append(e0.elapsed_time(e1) * 1000 / 20)
            base = sum(res[0]) / len(res[0])
            for R in rows:
                us = sum(res[R]) / len(res[R])
                mb = R * V * 2 / 1e6
                rate = "%.2f TB/s" % (mb * 1e6 / ((us - base) * 1e-6) / 1e12) if R and us > base else ""
                print("%s  n=%d  rows=%3d  %6.1f MB  %8.2f us  marginal %6.2f us  %s"
                      % (name, n, R, mb, us, us - base, rate), flush=True)
        del cache
        torch.cuda.empty_cache()


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    sub = ap.add_subparsers(dest="cmd", required=True)
    st = sub.add_parser("stream", help="run streamprobe (attn ... | evict ... | read ... | readpol ... | lanes)")
    st.add_argument("args", nargs=argparse.REMAINDER)
    en = sub.add_parser("entropy", help="entropy's marginal time in the fused base-attention launch")
    en.add_argument("--rows", default="0,1,8,32,64,128,256")
    a = ap.parse_args(argv)
    if a.cmd == "stream":
        if not os.path.exists(BIN):
            build()
        return subprocess.call([BIN] + a.args)
    rows = sorted({0} | {int(x) for x in a.rows.split(",")})
    entropy_marginal(rows)
    return 0


if __name__ == "__main__":
    sys.exit(main())
