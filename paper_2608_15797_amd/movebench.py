"""Timing of the fork / commit data movement on the 7B shape (App. C, the
fork-based engine; Alg. 1 retain / append-and-evict branches).

    python -m paper_2608_15797_amd.movebench [--P 16] [--N 8] [--B 512] [--buffer 128] [--T 128]

Measured per call, with HIP events over repeated launches on one stream:
  fork     P trajectory states with n = B + buffer live slots fanned out to
           P * N candidate caches (K, V, pos and the score row);
  append   T tokens appended to each of the P states (a committed helper
           step encoded in one pass);
  commit   append + window scores from the last W queries + TopB eviction
           of every state (the whole helper-accepted branch);
  prompt   one-shot compression of a T_prompt-token prompt to B (append,
           score, evict) for P sequences.
Algorithmic bytes: fork reads each source's live slots once and writes
every copy (sources fanned out to consecutive destinations share an L2
slice); append reads and writes the T rows. Both are plain copies, bound by
HBM bandwidth (8 TB/s nameplate).
"""
from __future__ import annotations

import argparse
import json
import math

import torch

from . import kvr, synth
from .workloads import QWEN7B


def _time(fn, reps):
    fn()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        fn()
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / reps


def measure(P=16, N=8, B=512, W=128, buffer=128, T=128, T_prompt=4096, seed=5):
    L, Hq, Hkv, D = QWEN7B["L"], QWEN7B["Hq"], QWEN7B["Hkv"], QWEN7B["D"]
    dt = torch.bfloat16
    esz = 2
    n = B + buffer
    cap_state = n + T + 1
    state = kvr.Cache.empty(P, L, Hkv, cap_state, D, dt)
    synth.fill_normal_(state.k, 1.0, seed, "mv", "k")
    synth.fill_normal_(state.v, 1.0, seed, "mv", "v")
    state.pos.copy_(torch.arange(cap_state, dtype=torch.int32, device="cuda"))
    ssc = torch.rand((P, L, Hkv, cap_state), device="cuda")
    cand = kvr.Cache.empty(P * N, L, Hkv, B + buffer + 1, D, dt)
    csc = torch.zeros((P * N, L, Hkv, B + buffer + 1), device="cuda")
    idx = (torch.arange(P * N, dtype=torch.int32, device="cuda") // N).contiguous()
    lens = torch.full((P * N,), n, dtype=torch.int32, device="cuda")
    row = 2 * D * esz + 4 + 4
    fork_bytes = (P + P * N) * L * Hkv * n * row
    t_fork = _time(lambda: kvr.fork(state, cand, idx, lens, ssc, csc), 20)

    # Append T tokens at live length n - T (so the state never overflows its cap).
    kn = synth.normal((P, L, Hkv, T, D), 1.0, seed, "mv", "kn", device="cuda", dtype=dt)
    vn = synth.normal((P, L, Hkv, T, D), 1.0, seed, "mv", "vn", device="cuda", dtype=dt)
    pn = torch.arange(T, dtype=torch.int32, device="cuda").repeat(P, 1).contiguous()
    n0 = torch.full((P,), B, dtype=torch.int32, device="cuda")
    app_bytes = 2 * P * L * Hkv * T * (2 * D * esz + 4)
    t_app = _time(lambda: kvr.append(state, n0, kn, vn, pn), 50)

    # Whole helper-accepted branch: append T at length B + buffer / 2, score, evict.
    scale = 1.0 / math.sqrt(D)
    pol = kvr.Policy(B, W, buffer)
    start = B + buffer // 2
    ln0 = torch.full((P,), start, dtype=torch.int32, device="cuda")
    ln1 = torch.full((P,), start + T, dtype=torch.int32, device="cuda")
    nq = min(W, T)
    qw = synth.normal((P, L, Hq, nq, D), 1.0, seed, "mv", "q", device="cuda", dtype=dt)
    sc = torch.zeros((P, L, Hkv, cap_state), device="cuda")

    def commit():
        kvr.append(state, ln0, kn, vn, pn)
        kvr.accumulate_scores(state, ln1, qw, scale, sc)
        kvr.evict_topb(state, ln1, sc, pol)

    t_commit = _time(commit, 20)
    t_score = _time(lambda: kvr.accumulate_scores(state, ln1, qw, scale, sc), 20)
    t_evict = _time(lambda: kvr.evict_topb(state, ln1, sc, pol), 20)
    del state, cand, ssc, csc, sc
    torch.cuda.empty_cache()

    # One-shot prompt compression.
    pc = kvr.Cache.empty(P, L, Hkv, T_prompt, D, dt)
    pk = synth.normal((P, L, Hkv, T_prompt, D), 1.0, seed, "mv", "pk", device="cuda", dtype=dt)
    pv = synth.normal((P, L, Hkv, T_prompt, D), 1.0, seed, "mv", "pv", device="cuda", dtype=dt)
    pp = torch.arange(T_prompt, dtype=torch.int32, device="cuda").repeat(P, 1).contiguous()
    zero = torch.zeros((P,), dtype=torch.int32, device="cuda")
    full = torch.full((P,), T_prompt, dtype=torch.int32, device="cuda")
    qp = synth.normal((P, L, Hq, W, D), 1.0, seed, "mv", "qp", device="cuda", dtype=dt)
    psc = torch.zeros((P, L, Hkv, T_prompt), device="cuda")

    def prompt():
        kvr.append(pc, zero, pk, pv, pp)
        kvr.accumulate_scores(pc, full, qp, scale, psc)
        kvr.evict_topb(pc, full, psc, pol)

    t_prompt = _time(prompt, 5)

    def gbps(b, ms):
        return round(b / (ms * 1e-3) / 1e9, 1)

    # Write-only reference: a 4 GiB fill kernel (fork is mostly writes).
    del pc, pk, pv, psc
    torch.cuda.empty_cache()
    big = torch.empty(1 << 31, dtype=torch.bfloat16, device="cuda")
    t_fill = _time(lambda: big.fill_(1.0), 10)
    fill_gbps = gbps(big.numel() * 2, t_fill)
    del big
    torch.cuda.empty_cache()

    return dict(
        shape=dict(P=P, N=N, L=L, Hq=Hq, Hkv=Hkv, D=D, B=B, W=W, buffer=buffer, T=T,
                   T_prompt=T_prompt, dtype="bf16"),
        fork=dict(us=round(t_fork * 1e3, 2), alg_bytes=fork_bytes, GBps=gbps(fork_bytes, t_fork),
                  frac=round(fork_bytes / (t_fork * 1e-3) / 8e12, 4)),
        append=dict(us=round(t_app * 1e3, 2), alg_bytes=app_bytes, GBps=gbps(app_bytes, t_app),
                    frac=round(app_bytes / (t_app * 1e-3) / 8e12, 4)),
        commit=dict(us=round(t_commit * 1e3, 2), score_us=round(t_score * 1e3, 2),
                    evict_us=round(t_evict * 1e3, 2)),
        prompt=dict(us=round(t_prompt * 1e3, 2)),
        fill_ref_GBps=fill_gbps,
    )


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--P", type=int, default=16)
    ap.add_argument("--N", type=int, default=8)
    ap.add_argument("--B", type=int, default=512)
    ap.add_argument("--window", type=int, default=128)
    ap.add_argument("--buffer", type=int, default=128)
    ap.add_argument("--T", type=int, default=128)
    ap.add_argument("--prompt", type=int, default=4096)
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        raise SystemExit("the movement measurement needs a GPU")
    print(json.dumps(measure(args.P, args.N, args.B, args.window, args.buffer, args.T,
                             args.prompt)), flush=True)


if __name__ == "__main__":
    main()
