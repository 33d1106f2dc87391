"""Per-step decode driver for the synthetic KV-Rescue workloads.

One step of the hot path for a batch of candidates (Eq. (3): the N base and N
helper candidates of every problem decode together) is:
  1. base:   kvr_decode_attn over the evicted cache, appending the new token
             and streaming the window importance score (Eq. (1), Sec. 2.1);
  2. base:   kvr_evict_topb when the live length exceeds B + buffer;
  3. helper: kvr_decode_attn over the shared or private full context plus the
             candidate's own suffix (Sec. 3.1);
  4. the entropies of the logit rows of both models, with the
             moving-average detector on the base rows (Eq. (4); only base
             candidates are screened): computed in the base-attention launch
             of step 1 (kvr_decode_attn_entropy) when the workload has a base
             model, else in the helper's context launch of step 3 (the same
             call with the prefix).

All candidates advance in lockstep, so every live length is known on the host
in advance: the driver precomputes per-token length tables on the device
(base: +1 per token, B after an eviction; helper suffix: 1 + t mod 512,
restarting after 512 tokens as if a step had been committed) and passes a
row of them to each call. No length ever travels back to the host.

Prompt tokens go through the same base loop (teacher forcing) before the
decode steps. Per-step inputs come from a pool of distinct seeded draws that
is cycled (large enough to exceed the 256 MB last-level cache), or one draw
per token when `per_token_inputs` is set (used for exact parity runs).
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional

import torch

from . import kvr, synth
from .workloads import Workload

POOL_BYTES = 512 << 20
MAX_POOL = 16


def base_length_schedule(T: int, B: int, buffer: int) -> list[int]:
    """Live length (after appending) of each token t < T, starting empty."""
    out, n = [], 0
    for _ in range(T):
        n += 1
        out.append(n)
        if n > B + buffer:
            n = B
    return out


def helper_suffix_schedule(T: int, scap: int) -> list[int]:
    return [1 + (t % scap) for t in range(T)]


@dataclass
class StepInputs:
    bq: Optional[torch.Tensor] = None
    bk: Optional[torch.Tensor] = None
    bv: Optional[torch.Tensor] = None
    hq: Optional[torch.Tensor] = None
    hk: Optional[torch.Tensor] = None
    hv: Optional[torch.Tensor] = None
    logits: tuple = ()


class Decoder:
    """Owns every device buffer of one workload and runs its steps."""

    def __init__(self, wl: Workload, device="cuda", per_token_inputs=False, pool=None,
                 gen_device=None, with_helper_prefix=True):
        self.wl = wl
        self.device = torch.device(device)
        self.dt = synth.torch_dtype(wl.dtype)
        b, h = wl.base, wl.helper
        self.T_prompt = b.prompt if b else 0
        self.T = self.T_prompt + wl.steps
        gen_device = gen_device or ("cpu" if per_token_inputs else self.device)
        dev = self.device

        if b:
            self.bcache = kvr.Cache.empty(b.S, b.L, b.Hkv, b.cache_cap, b.D, self.dt, dev)
            self.bcache.k.zero_()
            self.bcache.v.zero_()
            self.scores = torch.zeros((b.S, b.L, b.Hkv, b.cache_cap), dtype=torch.float32, device=dev)
            self.bout = torch.empty((b.S, b.L, b.Hq, b.D), dtype=self.dt, device=dev)
            self.policy = kvr.Policy(b.B, b.W, b.buffer)
            self.bscale = 1.0 / math.sqrt(b.D)
            self.blen_host = base_length_schedule(self.T, b.B, b.buffer)
            self.blen = torch.tensor(self.blen_host, dtype=torch.int32).repeat_interleave(b.S) \
                .view(self.T, b.S).to(dev)
            self.bpos = torch.arange(self.T, dtype=torch.int32).repeat_interleave(b.S) \
                .view(self.T, b.S).to(dev)
            self.kept = torch.empty((b.S, b.L, b.Hkv, b.B), dtype=torch.int32, device=dev)
        if h:
            if with_helper_prefix:
                pk, pv = synth.helper_prefix(wl, device=gen_device)
                self.prefix = kvr.Prefix(pk.to(dev), pv.to(dev))
            self.hcache = kvr.Cache.empty(h.S, h.L, h.Hkv, h.scap, h.D, self.dt, dev, with_pos=False)
            self.hcache.k.zero_()
            self.hcache.v.zero_()
            self.hout = torch.empty((h.S, h.L, h.Hq, h.D), dtype=self.dt, device=dev)
            self.hlen_host = helper_suffix_schedule(wl.steps, h.scap)
            self.hlen = torch.tensor(self.hlen_host, dtype=torch.int32).repeat_interleave(h.S) \
                .view(wl.steps, h.S).to(dev)
            wsb = kvr.decode_attn_workspace_size(self.hcache, self.prefix if with_helper_prefix else None,
                                                 h.Hq)
            self.hws = torch.empty(max(wsb, 16) // 4 + 4, dtype=torch.float32, device=dev)
        # Entropies ride in the base-attention launch when there is one, else
        # in the helper's context launch.
        self.fuse_entropy = bool(wl.logits)
        self.H = []
        self.ews = []
        for ls in wl.logits:
            self.H.append(torch.empty(ls.R, dtype=torch.float32, device=dev))
            n = kvr.logit_entropy_workspace_size(ls.R, ls.V)
            self.ews.append(torch.zeros(max(n, 16) // 4 + 4, dtype=torch.float32, device=dev))
        win, guard, tau = wl.detector
        # Only base candidates are screened (Sec. 3.2); helper rows get entropy only.
        self.detector = kvr.Detector.zeros(wl.logits[0].R, win, guard, tau, dev) \
            if (wl.logits and wl.base) else None
        # Workspace of the batched entropy call over every logit set.
        if wl.logits:
            n = kvr.logit_entropy_batch_workspace_size([(ls.R, ls.V) for ls in wl.logits], self.dt)
            self.ews_batch = torch.zeros(max(n, 16) // 4 + 4, dtype=torch.float32, device=dev)

        # Input pool.
        self.per_token = per_token_inputs
        if per_token_inputs:
            self.pool = [self._draw(t, gen_device) for t in range(self.T)]
        else:
            per = self._draw_bytes()
            P = pool or max(2, min(MAX_POOL, -(-POOL_BYTES // max(per, 1))))
            self.pool = [self._draw(i, gen_device) for i in range(P)]

    # -- inputs -------------------------------------------------------------
    def _draw_bytes(self) -> int:
        wl, es = self.wl, torch.tensor([], dtype=self.dt).element_size()
        n = 0
        if wl.base:
            b = wl.base
            n += b.S * b.L * (b.Hq + 2 * b.Hkv) * b.D * es
        if wl.helper:
            h = wl.helper
            n += h.S * h.L * (h.Hq + 2 * h.Hkv) * h.D * es
        for ls in wl.logits:
            n += ls.R * ls.V * es
        return n

    def _draw(self, idx: int, gen_device) -> StepInputs:
        wl, dev = self.wl, self.device
        si = StepInputs()
        if wl.base:
            si.bq, si.bk, si.bv = (x.to(dev) for x in synth.base_token(wl, idx, gen_device))
        if wl.helper:
            si.hq, si.hk, si.hv = (x.to(dev) for x in synth.helper_token(wl, idx, gen_device))
        si.logits = tuple(synth.logit_rows(wl, w, idx, gen_device).to(dev)
                          for w in range(len(wl.logits)))
        return si

    def inputs(self, t: int) -> StepInputs:
        return self.pool[t] if self.per_token else self.pool[t % len(self.pool)]

    # -- one token ------------------------------------------------------------
    def base_token(self, t: int, si: StepInputs, stream=None, on_scored=None,
                   timers=None, evict_log=None, only=None, sets=None) -> bool:
        """Append + attend (+ score) for token t; evict if the cache overflows.
        Returns True when an eviction ran. `on_scored(t)` (tests) runs between
        the attention and the eviction. With `evict_log` (a list), each
        eviction appends the number of kept rows, over all heads, that changed
        slot (read back from the kept sets: a synchronising copy, for
        accounting outside timed regions). With `sets` (LogitSet list) the
        entropies of those rows are computed in the same launch."""
        b = self.wl.base
        self.base_attn(t, si, stream, timers=timers, only=only, sets=sets)
        if on_scored is not None:
            on_scored(t)
        if self.blen_host[t] > b.B + b.buffer:
            with _timer(timers, "evict", stream, only):
                kvr.evict_topb(self.bcache, self.blen[t], self.scores, self.policy,
                               kept=self.kept, stream=stream)
            if evict_log is not None:
                slot = torch.arange(b.B, dtype=torch.int32, device=self.kept.device)
                evict_log.append(int((self.kept != slot).sum()))
            return True
        return False

    def base_attn(self, t: int, si: StepInputs, stream=None, timers=None, only=None, sets=None, sampler=None,
                  tokens=None) -> None:
        """The base-attention call of token t alone (append, attend, score),
        with the entropies of `sets` in the same launch when given, and with
        `sampler` the next token of every row into `tokens` (one tensor per
        set) as well."""
        if sets and sampler is not None:
            with _timer(timers, "base_attn_entropy_sample", stream, only):
                kvr.decode_attn_entropy_sample(self.bcache, self.blen[t], si.bq, self.bout, self.bscale, sets,
                                               sampler, tokens, k_new=si.bk, v_new=si.bv, new_pos=self.bpos[t],
                                               policy=self.policy, scores=self.scores, stream=stream)
        elif sets:
            with _timer(timers, "base_attn_entropy", stream, only):
                kvr.decode_attn_entropy(self.bcache, self.blen[t], si.bq, self.bout, self.bscale, sets,
                                        k_new=si.bk, v_new=si.bv, new_pos=self.bpos[t], policy=self.policy,
                                        scores=self.scores, stream=stream)
        else:
            with _timer(timers, "base_attn", stream, only):
                kvr.decode_attn(self.bcache, self.blen[t], si.bq, self.bout, self.bscale,
                                k_new=si.bk, v_new=si.bv, new_pos=self.bpos[t], policy=self.policy,
                                scores=self.scores, stream=stream)

    def helper_token(self, step: int, si: StepInputs, stream=None, timers=None, only=None, sets=None) -> None:
        """Helper attention of decode step `step`, with the entropies of
        `sets` (LogitSet list) in the context launch when given."""
        h = self.wl.helper
        if sets:
            with _timer(timers, "helper_attn_entropy", stream, only):
                kvr.decode_attn_entropy(self.hcache, self.hlen[step], si.hq, self.hout, h.softmax_scale, sets,
                                        k_new=si.hk, v_new=si.hv, prefix=self.prefix, workspace=self.hws,
                                        stream=stream)
            return
        with _timer(timers, "helper_attn", stream, only):
            kvr.decode_attn(self.hcache, self.hlen[step], si.hq, self.hout, h.softmax_scale,
                            k_new=si.hk, v_new=si.hv, prefix=self.prefix, workspace=self.hws,
                            stream=stream)

    def logit_sets(self, si: StepInputs) -> list:
        """The step's logit sets (the base set first, with the detector)."""
        return [kvr.LogitSet(lg, self.H[w], self.wl.logits[w].V,
                             detector=self.detector if w == 0 else None)
                for w, lg in enumerate(si.logits)]

    def entropy(self, si: StepInputs, stream=None, timers=None, only=None) -> None:
        """Entropies of every logit set of the step in one batched call."""
        if not si.logits:
            return
        sets = self.logit_sets(si)
        with _timer(timers, "entropy", stream, only):
            kvr.logit_entropy_batch(sets, workspace=self.ews_batch, stream=stream)

    def prompt(self, stream=None) -> None:
        for t in range(self.T_prompt):
            self.base_token(t, self.inputs(t), stream)

    def step(self, step: int, stream=None, timers=None, evict_log=None, only=None) -> None:
        """Decode step `step` (0-based, after the prompt): the whole hot path.
        With `timers` (a dict), each call (or only the call named `only`) is
        bracketed by a pair of timing events on the launch stream, appended
        under its name; `evict_log` as for base_token."""
        t = self.T_prompt + step
        si = self.inputs(t)
        fused = self.fuse_entropy and bool(si.logits)
        if self.wl.base:
            self.base_token(t, si, stream, timers=timers, evict_log=evict_log, only=only,
                            sets=self.logit_sets(si) if fused else None)
        if self.wl.helper:
            self.helper_token(step, si, stream, timers=timers, only=only,
                              sets=self.logit_sets(si) if fused and not self.wl.base else None)
        if not fused:
            self.entropy(si, stream, timers=timers, only=only)


class _timer:
    """Context manager recording start/end events around one library call
    (when timers is a dict and `only` is None or names this call)."""

    def __init__(self, timers, key, stream, only=None):
        self.timers = timers if (only is None or only == key) else None
        self.key, self.stream = key, stream

    def __enter__(self):
        if self.timers is not None:
            self.s = torch.cuda.Event(enable_timing=True)
            self.s.record(self.stream)
        return self

    def __exit__(self, *exc):
        if self.timers is not None:
            e = torch.cuda.Event(enable_timing=True)
            e.record(self.stream)
            self.timers.setdefault(self.key, []).append((self.s, e))
        return False
