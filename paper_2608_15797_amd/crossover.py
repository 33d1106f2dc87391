"""Evicted-vs-full decode crossover on MI355X (decode-compute analysis of the
appendix: per-token cost equations and the crossover l* = (1 + alpha) B').

    python -m paper_2608_15797_amd.crossover [--S 16] [--B 512] [--window 128] [--buffer 128]

Per decoded token and candidate, the attention side of decode costs:
  * full KV at context l: one attention pass over l cached tokens, C_attn(l),
    linear in l;
  * evicted: attention over at most B' = B + buffer cached tokens plus the
    eviction machinery, (1 + alpha) C_attn(B'), flat in l.
Evicted decode is cheaper once C_attn(l) exceeds (1 + alpha) C_attn(B').
The dense part of the model (2P per token) is the same on both sides and is
left out, so alpha and l* are comparable with the paper's figures while its
end-to-end speed-ups at 4k and 12k tokens (which include the dense part) are
not.

Everything is timed with the library's own kernels on the 7B shape (28 layers,
28 query / 4 KV heads, head_dim 128, bf16), S sequences per call:
  * full KV at several l, by both routes the library offers: the context
    (prefix) path with split-K over l, and the plain cache kernel over a cache
    of l tokens with scoring off; the faster one per l is used;
  * evicted, amortised: the average step over one whole eviction cycle of the
    policy as implemented here (lengths B+1 .. B+buffer+1; window scores
    streamed during the last W steps; one TopB eviction at the end);
  * evicted, per step: the cost model in which scoring and eviction run every
    step once l > B' (the setting the paper's alpha refers to): one scored
    attention step at B'+1 plus one TopB eviction; and the same with the
    redundancy-aware score (pooled importance mixed with key cosine
    similarity) computed before each eviction.
A least-squares line t(l) = a + b l is fitted to the full-KV times, then
  alpha = t_evict / t(B') - 1   and   l* = (t_evict - a) / b,
which is (1 + alpha) B' when the intercept a is small.
"""
from __future__ import annotations

import argparse
import json
import math
import sys

import torch

from . import kvr, synth
from .workloads import QWEN7B


def _time(fn, reps: int) -> float:
    """Average milliseconds of fn() over reps runs (after one warm-up run)."""
    fn()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        fn()
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / reps


def _qkv(S, L, Hq, Hkv, D, seed, tag):
    dt = torch.bfloat16
    return (synth.normal((S, L, Hq, D), 1.0, seed, tag, "q", device="cuda", dtype=dt),
            synth.normal((S, L, Hkv, D), 1.0, seed, tag, "k", device="cuda", dtype=dt),
            synth.normal((S, L, Hkv, D), 1.0, seed, tag, "v", device="cuda", dtype=dt))


def evicted_ms(S, L, Hq, Hkv, D, B, W, buffer, reps=3, seed=7):
    """(amortised ms/step over an eviction cycle, scored step at B'+1, one
    eviction call, unscored step at B') for the evicted base path."""
    cap = (B + buffer + 1 + 15) // 16 * 16  # heads 4 KiB-aligned, as the decode driver allocates
    cache = kvr.Cache.empty(S, L, Hkv, cap, D, torch.bfloat16)
    synth.fill_normal_(cache.k, 1.0, seed, "ev", "k")
    synth.fill_normal_(cache.v, 1.0, seed, "ev", "v")
    cache.pos.zero_()
    scores = torch.zeros((S, L, Hkv, cap), dtype=torch.float32, device="cuda")
    out = torch.empty((S, L, Hq, D), dtype=torch.bfloat16, device="cuda")
    q, kn, vn = _qkv(S, L, Hq, Hkv, D, seed, "ev")
    pol = kvr.Policy(B, W, buffer)
    lens = list(range(B + 1, B + buffer + 2))
    lent = torch.tensor(lens, dtype=torch.int32).repeat_interleave(S).view(len(lens), S).cuda()
    newpos = torch.zeros((S,), dtype=torch.int32, device="cuda")
    scale = 1.0 / math.sqrt(D)
    last = lent[-1]

    def step(i, scored=True):
        kvr.decode_attn(cache, lent[i], q, out, scale, k_new=kn, v_new=vn, new_pos=newpos,
                        policy=pol if scored else None, scores=scores if scored else None)

    def cycle():
        for i, n in enumerate(lens):
            step(i)
            if n > B + buffer:
                kvr.evict_topb(cache, lent[i], scores, pol)

    t_cycle = _time(cycle, reps) / len(lens)
    t_scored = _time(lambda: step(len(lens) - 1), 50)
    t_evict = _time(lambda: kvr.evict_topb(cache, last, scores, pol), 50)
    t_plain = _time(lambda: step(len(lens) - 2, scored=False), 50)
    mixed = torch.empty_like(scores)
    t_red = _time(lambda: kvr.redundancy_scores(cache, last, scores, pol, mixed), 50)
    del cache, scores, mixed
    torch.cuda.empty_cache()
    return t_cycle, t_scored, t_evict, t_plain, t_red


def full_ms(S, L, Hq, Hkv, D, ell, reps=10, seed=11):
    """(context path, cache kernel) ms per step of full-KV decode at context
    ell: ell-1 cached tokens plus the new one."""
    dt = torch.bfloat16
    q, kn, vn = _qkv(S, L, Hq, Hkv, D, seed, ell)
    out = torch.empty((S, L, Hq, D), dtype=dt, device="cuda")
    scale = 1.0 / math.sqrt(D)
    # Context path: private contexts of ell-1 tokens, own cache holds the new token.
    pk = torch.empty((S, L, Hkv, ell - 1, D), dtype=dt, device="cuda")
    pv = torch.empty_like(pk)
    synth.fill_normal_(pk, 1.0, seed, "full", ell, "k")
    synth.fill_normal_(pv, 1.0, seed, "full", ell, "v")
    prefix = kvr.Prefix(pk, pv)
    own = kvr.Cache.empty(S, L, Hkv, 16, D, dt, with_pos=False)
    ones = torch.ones((S,), dtype=torch.int32, device="cuda")
    ws = torch.empty(max(kvr.decode_attn_workspace_size(own, prefix, Hq), 16) // 4,
                     dtype=torch.float32, device="cuda")
    t_ctx = _time(lambda: kvr.decode_attn(own, ones, q, out, scale, k_new=kn, v_new=vn,
                                          prefix=prefix, workspace=ws), reps)
    del prefix, ws
    # Cache kernel: the same tokens in a cache of ell slots (no scoring).
    kc = torch.empty((S, L, Hkv, ell, D), dtype=dt, device="cuda")
    kc[..., : ell - 1, :].copy_(pk)
    del pk
    vc = torch.empty_like(kc)
    vc[..., : ell - 1, :].copy_(pv)
    del pv
    cache = kvr.Cache(kc, vc, None)
    lens = torch.full((S,), ell, dtype=torch.int32, device="cuda")
    t_cache = _time(lambda: kvr.decode_attn(cache, lens, q, out, scale, k_new=kn, v_new=vn), reps)
    del cache, kc, vc
    torch.cuda.empty_cache()
    return t_ctx, t_cache


def fit_line(xs, ys):
    n = len(xs)
    mx, my = sum(xs) / n, sum(ys) / n
    b = sum((x - mx) * (y - my) for x, y in zip(xs, ys)) / sum((x - mx) ** 2 for x in xs)
    return my - b * mx, b


def crossover_point(t, a, b, Bp, best):
    """Where evicted decode at t ms per step meets the fitted full-KV line
    t(l) = a + b l: alpha = t / t(B') - 1 and l* = (t - a) / b, with the
    speed-up over full KV at each measured length (best: l -> ms)."""
    t_bp = a + b * Bp
    return dict(ms=round(t, 5), alpha=round(t / t_bp - 1.0, 3),
                ell_star=round((t - a) / b, 1),
                speedup={str(k): round(v / t, 3) for k, v in best.items()})


def measure(S=16, B=512, W=128, buffer=128,
            lengths=(640, 1024, 2048, 3072, 4096, 6144, 8192, 12288, 16384)):
    L, Hq, Hkv, D = QWEN7B["L"], QWEN7B["Hq"], QWEN7B["Hkv"], QWEN7B["D"]
    t_cycle, t_scored, t_evict, t_plain, t_red = evicted_ms(S, L, Hq, Hkv, D, B, W, buffer)
    full = {}
    for ell in lengths:
        full[ell] = full_ms(S, L, Hq, Hkv, D, ell)
        print("# full KV l=%d: context path %.4f ms, cache kernel %.4f ms" % ((ell,) + full[ell]),
              file=sys.stderr, flush=True)
    best = {ell: min(v) for ell, v in full.items()}
    a, b = fit_line(list(best), list(best.values()))
    Bp = B + buffer
    t_bp = a + b * Bp
    t_step = t_scored + t_evict
    t_rkv = t_scored + t_red + t_evict

    def cross(t):
        return crossover_point(t, a, b, Bp, best)

    return dict(shape=dict(S=S, L=L, Hq=Hq, Hkv=Hkv, D=D, B=B, W=W, buffer=buffer, B_prime=Bp),
                full_ms={str(k): dict(context_path=round(v[0], 5), cache_kernel=round(v[1], 5))
                         for k, v in full.items()},
                fit=dict(intercept_ms=round(a, 5), ms_per_token=b, at_B_prime_ms=round(t_bp, 5)),
                parts_ms=dict(scored_step=round(t_scored, 5), eviction=round(t_evict, 5),
                              unscored_step=round(t_plain, 5), redundancy=round(t_red, 5)),
                evicted_amortised=cross(t_cycle), evicted_every_step=cross(t_step),
                evicted_every_step_redundancy=cross(t_rkv))


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--S", type=int, default=16)
    ap.add_argument("--B", type=int, default=512)
    ap.add_argument("--window", type=int, default=128)
    ap.add_argument("--buffer", type=int, default=128)
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        raise SystemExit("the crossover measurement needs a GPU")
    print(json.dumps(measure(args.S, args.B, args.window, args.buffer)), flush=True)


if __name__ == "__main__":
    main()
