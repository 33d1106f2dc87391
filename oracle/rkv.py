"""Oracle of the redundancy-aware eviction score (test infrastructure; only
tests/ and the benchmark's CPU leg use it).

The paper's evictor (App. C, KV eviction; Sec. 4.1; App. D.3) scores cached
tokens with a mix of query-attention importance and key redundancy measured by
cosine similarity, with mix weight lambda = 0.1, after pooling, and keeps the
top-B plus a protected recent window. It does not give the formula (that is
in the R-KV paper it cites). The reading implemented here, per (sequence,
layer, KV head) at an eviction with n live slots and candidates c < m = n - W:

  importance  I_c    = accumulated window attention of slot c (the score
                       row the decode path streams, Sec. 2.1);
  pooling     P_c    = max of I over the candidates within `pool // 2`
                       slots of c (1-D max pooling, clipped at the ends);
              Ih_c   = P_c / sum_c' P_c';
  redundancy  R_c    = mean cosine similarity of key c to the other
                       candidate keys = (1/(m-1)) sum_{c' != c} cos(k_c, k_c');
              Rh_c   = softmax over the candidates of R;
  score       Z_c    = lam * Ih_c - (1 - lam) * Rh_c,

and TopB of Eq. (1) selects on Z. A zero-norm key has cosine 0 with every
key. Parity of this composition against the paper is unpinned (the paper
has no formula); the pieces are pinned against their definitions'
consequences in tests/test_oracle_rkv.py.
fp64 throughout; bf16 keys are widened exactly.
"""
from __future__ import annotations

import numpy as np


def _widen(a) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def mean_cosine(keys) -> np.ndarray:
    """R_c for keys [m][D]: mean cosine similarity to the other m - 1 keys,
    by the plain pairwise definition."""
    k = _widen(keys)
    m = k.shape[0]
    if m < 2:
        return np.zeros(m)
    norms = np.sqrt((k * k).sum(axis=1))
    R = np.zeros(m)
    for c in range(m):
        tot = 0.0
        for d in range(m):
            if d == c or norms[c] == 0.0 or norms[d] == 0.0:
                continue
            tot += float(k[c] @ k[d]) / (norms[c] * norms[d])
        R[c] = tot / (m - 1)
    return R


def max_pool(I, pool: int) -> np.ndarray:
    I = np.asarray(I, dtype=np.float64)
    r = pool // 2
    m = len(I)
    return np.array([I[max(0, c - r): min(m, c + r + 1)].max() for c in range(m)])


def rkv_head(K_head, I_head, n: int, W: int, lam: float, pool: int) -> np.ndarray:
    """Z over the candidates c < n - W of one head (K_head [cap][D], I_head [cap])."""
    m = n - W
    P = max_pool(np.asarray(I_head, dtype=np.float64)[:m], pool)
    tot = P.sum()
    Ih = P / tot if tot > 0 else np.full(m, 1.0 / m)
    R = mean_cosine(np.asarray(K_head)[:m])
    e = np.exp(R - R.max())
    Rh = e / e.sum()
    return lam * Ih - (1.0 - lam) * Rh


def rkv_scores(K, I, n, W: int, lam: float, pool: int) -> np.ndarray:
    """Z[S][L][Hkv][cap] (zeros past each head's candidates) for caches
    K[S][L][Hkv][cap][D] and importance I[S][L][Hkv][cap]; n[S] live lengths."""
    S, L, Hkv, cap = np.asarray(I).shape
    Z = np.zeros((S, L, Hkv, cap))
    n = np.broadcast_to(np.asarray(n), (S,))
    for s in range(S):
        for l in range(L):
            for h in range(Hkv):
                Z[s, l, h, : n[s] - W] = rkv_head(K[s, l, h], I[s, l, h], int(n[s]), W, lam, pool)
    return Z
