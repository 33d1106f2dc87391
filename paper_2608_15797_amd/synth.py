"""Seeded synthetic inputs for the candidate-decode hot path.

This module is the one piece shared by the HIP path, the tests and the oracle
side of the tests. It draws random tensors and nothing else: it holds none of
the method's arithmetic (no attention, scores, selection or entropy).

Every tensor is keyed by a tuple (seed, name, indices...). The key is hashed
into a 63-bit seed for a fresh torch.Generator, so any slice of any workload
can be regenerated on its own. Values are drawn in fp32 and then rounded to
the storage dtype with round-to-nearest-even (torch's conversion).

Note: torch's CPU and GPU generators produce different streams for the same
seed. Tests that compare the GPU path against the oracle therefore always
download the exact device tensors the kernels consumed; they never regenerate
them on the other device.
"""
from __future__ import annotations

import hashlib
from typing import Sequence

import torch

_STD_NORMAL_CHUNK = 1 << 26  # elements per randn call when filling large buffers


def key_seed(*key) -> int:
    """63-bit generator seed derived from an arbitrary key tuple."""
    h = hashlib.sha256(repr(tuple(key)).encode()).digest()
    return int.from_bytes(h[:8], "little") & ((1 << 63) - 1)


def _gen(device, *key) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(key_seed(*key))
    return g


def normal(shape: Sequence[int], std: float, *key, device="cpu",
           dtype=torch.float32) -> torch.Tensor:
    """i.i.d. N(0, std^2) (std is the standard deviation), rounded to dtype."""
    g = _gen(device, *key)
    x = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(dtype)


def fill_normal_(out: torch.Tensor, std: float, *key) -> torch.Tensor:
    """Fill `out` with N(0, std^2) slice by slice along dim 0 (and dim 1 when a
    slice is large), so multi-GB buffers never need an fp32 copy in memory.
    Slice (i, j) is keyed by key + (i, j)."""
    assert out.dim() >= 2
    per_i = out[0].numel()
    for i in range(out.shape[0]):
        if per_i <= _STD_NORMAL_CHUNK:
            out[i].copy_(normal(out[i].shape, std, *key, i, device=out.device,
                                dtype=out.dtype))
        else:
            for j in range(out.shape[1]):
                out[i, j].copy_(normal(out[i, j].shape, std, *key, i, j,
                                       device=out.device, dtype=out.dtype))
    return out


def boosted_logits(R: int, V: int, std: float, n_boost: int, boost: float, *key,
                   device="cpu", dtype=torch.bfloat16, ld: int | None = None,
                   near_uniform_rows: Sequence[int] = (), near_uniform_std: float = 0.1
                   ) -> torch.Tensor:
    """Logit rows: N(0, std^2) with `n_boost` distinct uniformly chosen entries per
    row raised by `boost` (added in fp32 before rounding). Rows listed in
    `near_uniform_rows` are instead N(0, near_uniform_std^2) with no boost.
    Returns an [R, ld] tensor whose first V columns hold the row (ld >= V; the
    padding columns are zero)."""
    ld = V if ld is None else ld
    assert ld >= V
    x = normal((R, V), std, *key, "logits", device=device, dtype=torch.float32)
    if n_boost > 0:
        u = torch.rand((R, V), generator=_gen(device, *key, "boost_idx"),
                       device=device, dtype=torch.float32)
        idx = torch.topk(u, n_boost, dim=1).indices
        del u
        x.scatter_add_(1, idx, torch.full(idx.shape, float(boost), device=device))
    for r in near_uniform_rows:
        x[r] = normal((V,), near_uniform_std, *key, "near_uniform", r,
                      device=device, dtype=torch.float32)
    out = torch.zeros((R, ld), device=device, dtype=dtype)
    out[:, :V] = x.to(dtype)
    return out


def choose_rows(R: int, count: int, *key) -> list[int]:
    """A seeded set of `count` distinct row indices in [0, R)."""
    g = _gen("cpu", *key, "rows")
    return sorted(torch.randperm(R, generator=g)[:count].tolist())


# ---------------------------------------------------------------------------
# Per-token inputs of a workload. `idx` names the draw: the decode driver uses
# a pool of distinct draws and cycles through it; the tiny workload uses one
# draw per token.

def torch_dtype(name: str):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def base_token(wl, idx: int, device="cpu"):
    """(q[S][L][Hq][D], k[S][L][Hkv][D], v[S][L][Hkv][D]) of the base model."""
    b, dt = wl.base, torch_dtype(wl.dtype)
    q = normal((b.S, b.L, b.Hq, b.D), wl.qkv_std, wl.seed, "base_q", idx, device=device, dtype=dt)
    k = normal((b.S, b.L, b.Hkv, b.D), wl.qkv_std, wl.seed, "base_k", idx, device=device, dtype=dt)
    v = normal((b.S, b.L, b.Hkv, b.D), wl.qkv_std, wl.seed, "base_v", idx, device=device, dtype=dt)
    return q, k, v


def helper_token(wl, idx: int, device="cpu"):
    """(q[S][L][Hq][D], k[S][L][Hkv][D], v[S][L][Hkv][D]) of the helper model."""
    h, dt = wl.helper, torch_dtype(wl.dtype)
    q = normal((h.S, h.L, h.Hq, h.D), wl.qkv_std, wl.seed, "help_q", idx, device=device, dtype=dt)
    k = normal((h.S, h.L, h.Hkv, h.D), h.k_std, wl.seed, "help_k", idx, device=device, dtype=dt)
    v = normal((h.S, h.L, h.Hkv, h.D), wl.qkv_std, wl.seed, "help_v", idx, device=device, dtype=dt)
    return q, k, v


def helper_prefix(wl, device="cpu"):
    """Shared/private full-context prefixes K,V[P][L][Hkv][plen][D]."""
    h, dt = wl.helper, torch_dtype(wl.dtype)
    shape = (h.P, h.L, h.Hkv, h.plen, h.D)
    K = torch.empty(shape, device=device, dtype=dt)
    V = torch.empty(shape, device=device, dtype=dt)
    fill_normal_(K, h.k_std, wl.seed, "prefix_k")
    fill_normal_(V, wl.qkv_std, wl.seed, "prefix_v")
    return K, V


def logit_rows(wl, which: int, idx: int, device="cpu", ld=None):
    """Logits [R][ld] of model `which` (0 = base, 1 = helper) for draw idx."""
    ls = wl.logits[which]
    dt = torch_dtype(wl.dtype)
    nu = choose_rows(ls.R, int(-(-ls.near_uniform_frac * ls.R // 1)), wl.seed, "nu", which) \
        if ls.near_uniform_frac > 0 else ()
    return boosted_logits(ls.R, ls.V, ls.std, ls.n_boost, ls.boost, wl.seed, "logits",
                          which, idx, device=device, dtype=dt, ld=ld, near_uniform_rows=nu)
