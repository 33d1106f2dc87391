"""Oracle of the fork / commit data movement around the hot loop (test
infrastructure; only tests/ and the benchmark's CPU leg use it).

The fork-based engine of the implementation section keeps one persistent
trajectory state per problem. Each reasoning step
  * forks N base candidates by copying the live (post-eviction) KV slots of
    the state into fresh candidate slots;
  * when a base candidate wins, that candidate's cache becomes the new state
    (Alg. 1: retain the selected base fork) -- again a copy of live slots;
  * when a helper candidate wins, the base encodes the step's tokens in one
    forward pass: they are appended in bulk, scored from the queries of that
    pass, and the cache is evicted if it overflows (Alg. 1: append s_t to K_b
    and apply E_B). The same three moves compress a prompt in one shot.

Readings used (the paper names these moves but gives no formula for them):
  * a fork copies K, V, positions and the stored score row of the first
    `length` slots of every (layer, KV head); slots beyond are left as they
    were in the destination;
  * the importance of a one-pass commit is recomputed from the last
    min(W, T) queries of the T appended tokens, each attending causally
    (the observation window of Sec. 2.1 restricted to the queries that pass
    computes); eviction then follows Eq. (1) with that score when the
    length exceeds B + buffer.
Plain loops and numpy indexing; no blocking or reordering.
"""
from __future__ import annotations

import numpy as np

from . import compact_head, select_topb, window_scores


def fork(src: dict, dst: dict, src_index, length) -> None:
    """In-place on dst. src/dst: dicts with K, V [S][L][Hkv][cap][D] and
    optional pos [S][L][Hkv][cap], score [S][L][Hkv][cap]. For every
    destination s with src_index[s] >= 0, slots [0, length[s]) of source
    sequence src_index[s] are copied. Sources are read before any write, so
    src may be dst."""
    snap = {k: (None if v is None else v.copy()) for k, v in src.items()}
    for s in range(dst["K"].shape[0]):
        r = int(src_index[s])
        if r < 0:
            continue
        n = int(length[s])
        for key in ("K", "V", "pos", "score"):
            if dst.get(key) is None or snap.get(key) is None:
                continue
            for l in range(dst[key].shape[1]):
                for h in range(dst[key].shape[2]):
                    for j in range(n):
                        dst[key][s, l, h, j] = snap[key][r, l, h, j]


def append(cache: dict, length, k_new, v_new, pos_new=None) -> None:
    """In-place bulk append: token i of sequence s goes to slot length[s] + i
    of every (layer, KV head). k_new, v_new [S][L][Hkv][T][D]; pos_new [S][T]."""
    S, L, Hkv, T = k_new.shape[:4]
    for s in range(S):
        n = int(length[s])
        for l in range(L):
            for h in range(Hkv):
                for i in range(T):
                    cache["K"][s, l, h, n + i] = k_new[s, l, h, i]
                    cache["V"][s, l, h, n + i] = v_new[s, l, h, i]
                    if pos_new is not None and cache.get("pos") is not None:
                        cache["pos"][s, l, h, n + i] = pos_new[s, i]


def commit(cache: dict, n0: int, k_new, v_new, pos_new, q_step, scale: float,
           B: int, W: int, buffer: int):
    """One-pass commit of T tokens to every sequence (all at live length n0).
    q_step [S][L][Hq][T][D]: the queries of the T tokens. Returns (new live
    length, score [S][L][Hkv][cap] float64, kept [S][L][Hkv][B] or None)."""
    S, L, Hkv = k_new.shape[:3]
    T = k_new.shape[3]
    append(cache, [n0] * S, k_new, v_new, pos_new)
    n = n0 + T
    nq = min(W, T)
    score = window_scores(cache["K"], cache["V"], n, q_step[:, :, :, T - nq:], scale)
    if n <= B + buffer:
        return n, score, None
    kept = np.zeros((S, L, Hkv, B), np.int32)
    for s in range(S):
        for l in range(L):
            for h in range(Hkv):
                kept[s, l, h] = select_topb(score[s, l, h], n, B, W)
                pos = cache["pos"][s, l, h] if cache.get("pos") is not None else \
                    np.zeros(cache["K"].shape[3], np.int32)
                compact_head(cache["K"][s, l, h], cache["V"][s, l, h], pos, kept[s, l, h])
    return B, score, kept
