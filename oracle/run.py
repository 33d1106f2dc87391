"""Oracle of the evicted base model's per-token loop (test infrastructure).

Per token, for every candidate sequence (all advance in lockstep):
  1. append (k_t, v_t, t) at slot n, n <- n + 1            (C_t grows, Sec. 2.1)
  2. attend over the n live entries                       (Eq. (1), third line)
  3. if the token lies in the observation window, keep its per-KV-head
     attention-mass row (summed over the G query heads of the head)
  4. if n > B + buffer: score = sum of the window rows (accumulated
     attention, Sec. 2.1); keep the W newest entries plus the B - W
     best-scoring older ones (TopB of Eq. (1)); compact K, V, pos;
     n <- B; forget the window rows                       (Eq. (1), first two lines)

Readings of the paper used here (it gives no formula for the score and
describes the budget two ways):
  * after an eviction exactly B entries remain, W of them the protected
    recent window; the physical bound is B + buffer + 1;
  * the importance score is the sum, over the last W query positions, of the
    softmax probabilities of the G query heads sharing the KV head;
  * the observation window and the protected window have the same length W;
  * each (sequence, layer, KV head) selects its own kept set;
  * ties go to the lower slot; kept entries keep their temporal order;
  * prompt tokens go through the same loop (teacher forcing).
A window row of length-n step covers the slots that exist at that step and
is zero for slots appended later.
"""
from __future__ import annotations

import numpy as np

from . import compact_head, decode_attn, select_topb


def window_start(B: int, W: int, buffer: int) -> int:
    """Smallest live length n (after appending) whose step is in the window."""
    return B + buffer + 2 - W


class BaseOracle:
    """fp64 state machine for S lockstep candidate sequences."""

    def __init__(self, S, L, Hkv, Hq, D, B, W, buffer, dtype_np, scale, cap=None,
                 record_pre=False):
        assert 0 < W < B and buffer >= W - 1, "window rows must all follow the last eviction"
        self.S, self.L, self.Hkv, self.Hq, self.D = S, L, Hkv, Hq, D
        self.B, self.W, self.buffer = B, W, buffer
        self.cap = B + buffer + 1 if cap is None else cap
        assert self.cap >= B + buffer + 1
        self.scale = scale
        self.K = np.zeros((S, L, Hkv, self.cap, D), dtype_np)
        self.V = np.zeros((S, L, Hkv, self.cap, D), dtype_np)
        self.pos = np.full((S, L, Hkv, self.cap), -1, np.int32)
        self.n = 0
        self.rows = []          # window rows, each [S][L][Hkv][cap]
        self.events = []        # one dict per eviction
        self.record_pre = record_pre

    def step(self, t, q, k, v):
        """One token. q[S][L][Hq][D], k,v[S][L][Hkv][D]. Returns out float64."""
        assert self.n < self.cap
        self.K[:, :, :, self.n] = k
        self.V[:, :, :, self.n] = v
        self.pos[:, :, :, self.n] = t
        self.n += 1
        out, psum = decode_attn(self.K, self.V, self.n, q, self.scale)
        if self.n >= window_start(self.B, self.W, self.buffer):
            self.rows.append(psum)
        if self.n > self.B + self.buffer:
            self.evict(t)
        return out

    def evict(self, t):
        n = self.n
        assert len(self.rows) == self.W, "window rows %d != W" % len(self.rows)
        score = np.sum(self.rows, axis=0)
        kept = np.zeros((self.S, self.L, self.Hkv, self.B), np.int32)
        for s in range(self.S):
            for l in range(self.L):
                for h in range(self.Hkv):
                    kept[s, l, h] = select_topb(score[s, l, h], n, self.B, self.W)
        kept_pos = np.take_along_axis(self.pos, kept, axis=3)
        pre = (self.K.copy(), self.V.copy(), self.pos.copy()) if self.record_pre else None
        for s in range(self.S):
            for l in range(self.L):
                for h in range(self.Hkv):
                    compact_head(self.K[s, l, h], self.V[s, l, h], self.pos[s, l, h],
                                 kept[s, l, h])
        self.events.append(dict(t=t, n=n, score=score[..., :n].copy(), kept=kept,
                                kept_pos=kept_pos, pre=pre))
        self.n = self.B
        self.rows = []


def min_pairwise_gap(score_row, n, W):
    """Smallest gap between any two candidate (non-window) scores of one head."""
    c = np.sort(np.asarray(score_row[: n - W], dtype=np.float64))
    return float(np.min(np.diff(c))) if len(c) > 1 else np.inf


def boundary_gap(score_row, n, B, W):
    """Gap between the (B-W)-th and (B-W+1)-th largest candidate scores."""
    c = np.sort(np.asarray(score_row[: n - W], dtype=np.float64))[::-1]
    k = B - W
    return float(c[k - 1] - c[k]) if len(c) > k else np.inf
