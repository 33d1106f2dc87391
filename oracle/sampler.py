"""Oracle of the per-token sampler fused with the entropy pass (test
infrastructure; only tests/ and the benchmark's CPU leg use it).

Decoding samples at temperature 0.8 with top-k 20 and top-p 0.95 (Sec. 4.1
decoding setup; App. C, decoding and evaluation). The paper names the three
settings but not their order or tie rules; the reading used here is the
common one:
  1. scale the logits by 1 / temperature;
  2. keep the top_k largest logits (ties to the lower token id);
  3. softmax over those k, sorted by probability, descending (ties to the
     lower token id);
  4. keep the shortest prefix of that order whose cumulative probability is
     at least top_p (always at least one token);
  5. draw one token from the kept prefix, renormalised, by inverse CDF with a
     uniform u in [0, 1): the first token whose cumulative mass exceeds
     u times the prefix mass.
The uniform comes from a counter-based generator, so that host and device
draw the same u: Philox4x64-10 (Salmon, Moraes, Dror and Shaw, "Parallel
random numbers: as easy as 1, 2, 3", SC 2011), counter (step, row, 0, 0),
key (seed, 0), first output word, top 24 bits: u = (w0 >> 40) / 2^24.
fp64 throughout; bf16 logits are widened exactly.
"""
from __future__ import annotations

import numpy as np

_M64 = (1 << 64) - 1
# Philox4x64 multipliers and Weyl key increments (published constants).
_PH_M0, _PH_M1 = 0xD2E7470EE14C6C93, 0xCA5A826395121157
_PH_W0, _PH_W1 = 0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B


def philox4x64_10(ctr, key):
    """Ten Philox rounds on a 4 x 64-bit counter with a 2 x 64-bit key."""
    c = [int(x) & _M64 for x in ctr]
    k = [int(x) & _M64 for x in key]
    for _ in range(10):
        p0 = _PH_M0 * c[0]
        p1 = _PH_M1 * c[2]
        c = [((p1 >> 64) ^ c[1] ^ k[0]) & _M64, p1 & _M64,
             ((p0 >> 64) ^ c[3] ^ k[1]) & _M64, p0 & _M64]
        k = [(k[0] + _PH_W0) & _M64, (k[1] + _PH_W1) & _M64]
    return c


def uniform(seed: int, step: int, row: int) -> float:
    """24-bit uniform in [0, 1) of (seed, step, row)."""
    w0 = philox4x64_10((step, row, 0, 0), (seed, 0))[0]
    return (w0 >> 40) / float(1 << 24)


def _widen(row) -> np.ndarray:
    a = np.asarray(row)
    if a.dtype == np.uint16:                       # raw bf16 bits
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def sample_row(logits, V: int, temperature: float, top_k: int, top_p: float, u: float):
    """Returns (token, detail). detail holds the sorted candidate ids, their
    renormalised top-k probabilities, the prefix length kept by top-p, and the
    smallest distance of a decision from its threshold (cumulative mass vs
    top_p, and vs u times the prefix mass), for tests that must tell a
    rounding-sensitive draw from a wrong one."""
    x = _widen(logits)[:V]
    k = min(top_k, V)
    order = np.lexsort((np.arange(V), -x))[:k]     # value desc, then id asc
    z = x[order] / temperature
    if not np.isfinite(z[0]):
        raise ValueError("row has no finite logit")
    w = np.exp(z - z[0])
    q = w / w.sum()
    cum = np.cumsum(q)
    keep = int(np.argmax(cum >= top_p)) + 1 if top_p < 1.0 and np.any(cum >= top_p) else k
    mass = cum[keep - 1]
    target = u * mass
    pick = int(np.argmax(cum[:keep] > target)) if np.any(cum[:keep] > target) else keep - 1
    margin_p = float(np.min(np.abs(cum[:k] - top_p))) if top_p < 1.0 else np.inf
    margin_u = float(np.min(np.abs(cum[:keep] - target)))
    return int(order[pick]), dict(order=order, q=q, keep=keep, margin_p=margin_p,
                                  margin_u=margin_u, pick=pick)


def sample(logits, V: int, temperature: float, top_k: int, top_p: float, seed: int, step: int):
    """Tokens [R] and per-row details for logits [R][>=V]."""
    toks, det = [], []
    for r in range(logits.shape[0]):
        t, d = sample_row(logits[r], V, temperature, top_k, top_p, uniform(seed, step, r))
        toks.append(t)
        det.append(d)
    return np.array(toks, np.int32), det
