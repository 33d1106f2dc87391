"""Host-side plan of the benchmark: which decode steps it times and the
algorithmic bytes of each call of those steps (no GPU work here).

Lengths and inputs are functions of the decode step index (all candidates
advance in lockstep), so a timed window can be any K consecutive step
indices; place_window puts an eviction and the observation-window steps
before it inside the window.
"""
from __future__ import annotations

from . import accounting as acc
from .pipeline import base_length_schedule, helper_suffix_schedule

PEAK_HBM_GBPS = 8000.0


def cycle_steps(wl) -> int:
    """Steps of one whole cycle: whole eviction periods (buffer + 1 steps)
    covering the helper's 512-token suffix cycle (or 512 steps for a
    base-only workload); the suffix cycle alone for a helper-only one."""
    b, h = wl.base, wl.helper
    span = h.scap if h else 512
    if not b:
        return span
    pb = b.buffer + 1
    return pb * (-(-span // pb))


class Schedule:
    """Live lengths of every decode step index, as the decode driver computes
    them (base: +1 per token, B after an eviction; helper suffix 1 + i mod 512)."""

    def __init__(self, wl, horizon, fuse_entropy=None):
        self.wl = wl
        b, h = wl.base, wl.helper
        # As the decode driver: entropies in the base-attention launch, or in
        # the helper's context launch when there is no base model.
        self.fuse_entropy = bool(wl.logits) if fuse_entropy is None else fuse_entropy
        self.T_prompt = b.prompt if b else 0
        self.blen_host = base_length_schedule(self.T_prompt + horizon, b.B, b.buffer) if b else None
        self.hlen_host = helper_suffix_schedule(horizon, h.scap) if h else None

    def base_n(self, i):
        return self.blen_host[self.T_prompt + i]

    def evicts(self, i):
        b = self.wl.base
        return b is not None and self.base_n(i) > b.B + b.buffer

    def scores(self, i):
        b = self.wl.base
        return b is not None and self.base_n(i) >= b.B + b.buffer + 2 - b.W


def place_window(wl, K, W, horizon=None):
    """First decode step index s0 of the K timed steps (see the module
    docstring); s0 >= W so that the warmup steps exist."""
    b, h = wl.base, wl.helper
    C = cycle_steps(wl)
    horizon = horizon or (W + K + 3 * C)
    sch = Schedule(wl, horizon)
    suf_mean = (h.scap + 1) / 2.0 if h else None
    if b:
        lead = min(b.W - 1, K - 1)
        best = None
        for e in range(horizon - K):
            if not sch.evicts(e):
                continue
            s0 = e - lead
            if s0 < W:
                continue
            if e > W + lead + C and best is not None:
                break
            cost = 0.0 if not h else abs(sum(sch.hlen_host[s0:s0 + K]) / K - suf_mean)
            if best is None or cost < best[0]:
                best = (cost, s0)
        assert best is not None, "no eviction fits the window"
        return best[1]
    # Helper only: centre the window on the suffix cycle.
    s0 = max(W, int(round(suf_mean - (K + 1) / 2.0)))
    return s0


def cycle_start(wl, after):
    """First step index >= after where a whole cycle starts: the step after an
    eviction (base live length B + 1), else a suffix restart."""
    b, h = wl.base, wl.helper
    sch = Schedule(wl, after + 2 * cycle_steps(wl) + 2)
    i = after
    if b:
        while sch.base_n(i) != b.B + 1:
            i += 1
        return i
    while sch.hlen_host[i] != 1:
        i += 1
    return i


def window_stats(wl, sch, s0, K):
    """What the K steps from s0 contain (evictions, score steps, mean lengths)."""
    out = dict(first_step=s0, steps=K)
    if wl.base:
        out["evictions_in_window"] = sum(sch.evicts(i) for i in range(s0, s0 + K))
        out["score_steps_in_window"] = sum(sch.scores(i) for i in range(s0, s0 + K))
        out["mean_base_len"] = round(sum(sch.base_n(i) for i in range(s0, s0 + K)) / K, 2)
    if wl.helper:
        out["mean_helper_suffix"] = round(sum(sch.hlen_host[s0:s0 + K]) / K, 2)
    return out


def step_bytes(wl, dec, i, moved_rows=None):
    """Algorithmic bytes of decode step i by call name. moved_rows: kept rows
    per head that change slot at an eviction, on average (None = all B, the
    upper bound). When the decoder computes the entropies inside an attention
    launch (dec.fuse_entropy), that call is "base_attn_entropy" (with a base
    model) or "helper_attn_entropy" (helper only) and carries the logit bytes
    too."""
    out = {}
    fused = getattr(dec, "fuse_entropy", False) and bool(wl.logits)
    if wl.base:
        b = wl.base
        n = dec.blen_host[dec.T_prompt + i]
        if fused:
            out["base_attn_entropy"] = acc.base_attn_bytes(wl, n) + acc.entropy_bytes(wl)
        else:
            out["base_attn"] = acc.base_attn_bytes(wl, n)
        if n > b.B + b.buffer:
            out["evict"] = acc.evict_bytes(wl, n, moved_rows)
    if wl.helper:
        if fused and not wl.base:
            out["helper_attn_entropy"] = acc.helper_attn_bytes(wl, dec.hlen_host[i]) + acc.entropy_bytes(wl)
        else:
            out["helper_attn"] = acc.helper_attn_bytes(wl, dec.hlen_host[i])
    if wl.logits and not fused:
        out["entropy"] = acc.entropy_bytes(wl)  # every logit set, one batched call
    return out


def window_bytes(wl, dec, steps, moved_rows=None):
    tot = {}
    for i in steps:
        for k, v in step_bytes(wl, dec, i, moved_rows).items():
            tot[k] = tot.get(k, 0) + v
    return tot


def dominant_call(wl, dec, steps):
    tot = window_bytes(wl, dec, steps)
    return max(tot, key=tot.get)
