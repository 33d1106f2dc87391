"""Algorithmic HBM bytes and flops of each hot-path call (host arithmetic).

Algorithmic bytes are what the method itself must move, independent of the
kernels' blocking:
  base attention  K and V of the n live entries (the new token's row read once
                  and written once), q read, o written, the new position written,
                  and the score row read+written in window steps (written only
                  in the first window step);
  eviction        the n - W candidate scores read, the kept rows of K and V that
                  change slot read and written (upper bound: all B rows), pos
                  likewise;
  helper          every prefix's K and V once per step (shared prefixes are
                  counted once, not once per candidate), each candidate's suffix
                  rows, q read, o written;
  entropy         R x V logits read, R entropies written (detector state is a
                  few bytes per row and is ignored).
Flops: 4 * D * n per query row and key span (q.k and p.v), the attention term
4 L d l of the overhead-derivation appendix with l = n.
"""
from __future__ import annotations

from .workloads import Workload


def esize(wl: Workload) -> int:
    return 4 if wl.dtype == "f32" else 2


def base_attn_bytes(wl: Workload, n: int) -> int:
    b, e = wl.base, esize(wl)
    heads = b.S * b.L * b.Hkv
    kv = heads * (n + 1) * 2 * b.D * e           # n rows read + the new row written
    qo = b.S * b.L * b.Hq * b.D * e * 2
    pos = b.S * b.L * b.Hkv * 4
    wstart = b.B + b.buffer + 2 - b.W
    sc = 0
    if n >= wstart:
        sc = heads * n * 4 * (1 if n == wstart else 2)
    return kv + qo + pos + sc


def base_attn_flops(wl: Workload, n: int) -> int:
    b = wl.base
    return 4 * b.D * n * b.S * b.L * b.Hq


def evict_bytes(wl: Workload, n: int, moved_rows: float | None = None) -> int:
    """moved_rows: kept rows per head that change slot, on average over the
    heads (None = the upper bound, all B)."""
    b, e = wl.base, esize(wl)
    heads = b.S * b.L * b.Hkv
    m = b.B if moved_rows is None else moved_rows
    return int(heads * ((n - b.W) * 4 + m * 2 * (2 * b.D * e + 4)))


def helper_attn_bytes(wl: Workload, u: int) -> int:
    """u = suffix length including the new token."""
    h, e = wl.helper, esize(wl)
    pre = h.P * h.L * h.Hkv * h.plen * 2 * h.D * e
    suf = h.S * h.L * h.Hkv * (u + 1) * 2 * h.D * e
    qo = h.S * h.L * h.Hq * h.D * e * 2
    return pre + suf + qo


def helper_attn_flops(wl: Workload, u: int) -> int:
    h = wl.helper
    return 4 * h.D * (h.plen + u) * h.S * h.L * h.Hq


def entropy_bytes(wl: Workload) -> int:
    e = esize(wl)
    return sum(ls.R * ls.V * e + ls.R * 4 for ls in wl.logits)
