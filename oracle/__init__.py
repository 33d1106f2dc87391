"""CPU oracle for the KV-Rescue candidate-decode hot path (test infrastructure).

Only tests/, the smoke check and the benchmark's CPU-baseline leg may import
this package. The product path never does, and this package imports nothing
from the product (it takes plain numpy arrays).

The arithmetic lives in kvr_oracle.c (fp64, plain loops); this file builds it
with gcc, loads it with ctypes and converts arrays. bf16 arrays are passed as
their raw uint16 bit patterns.

Pinned by tests/test_oracle_*.py against brute force, closed forms,
library routines and invariants (see the docstrings there).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kvr_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

F32, BF16 = 0, 1


def build(force: bool = True) -> str:
    """Compile kvr_oracle.c into liboracle.so (gcc, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        vp, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_long, ctypes.c_double
        L.orc_decode_attn.argtypes = [vp, vp, i32, i32, i32, i32, i32, i32, vp, vp, i32, i32,
                                      vp, vp, i32, f64, vp, vp]
        L.orc_window_scores.argtypes = [vp, vp, i32, i32, i32, i32, i32, i32, vp, vp, i32,
                                        i32, f64, vp]
        L.orc_select_topb.argtypes = [vp, i32, i32, i32, vp]
        L.orc_compact_head.argtypes = [vp, vp, vp, i32, i32, vp, i32]
        L.orc_entropy.argtypes = [vp, i32, i32, i32, i64, f64, vp]
        L.orc_detector_step.argtypes = [vp, i32, vp, vp, vp, i32, i32, f64]
        for f in (L.orc_decode_attn, L.orc_window_scores, L.orc_select_topb,
                  L.orc_compact_head, L.orc_entropy, L.orc_detector_step):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def set_threads(n: int) -> None:
    """OpenMP thread count used by the oracle (a reported baseline knob)."""
    os.environ["OMP_NUM_THREADS"] = str(n)
    try:
        ctypes.CDLL("libgomp.so.1").omp_set_num_threads(ctypes.c_int(n))
    except OSError:
        pass


def threads() -> int:
    try:
        return int(ctypes.CDLL("libgomp.so.1").omp_get_max_threads())
    except OSError:
        return 1


def _dt(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    raise TypeError("oracle inputs are float32 or bf16 bit patterns (uint16), got %s" % a.dtype)


def _c(a):
    return np.ascontiguousarray(a)


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc, what):
    if rc != 0:
        raise ValueError("oracle %s rejected its arguments (rc=%d)" % (what, rc))


def decode_attn(K, V, n, q, scale, prefix_K=None, prefix_V=None, want_psum=True):
    """Attention of q[S][L][Hq][D] over cache K,V[S][L][Hkv][cap][D] (n[s] live
    entries) and an optional shared prefix [P][L][Hkv][plen][D].
    Returns (out[S][L][Hq][D] float64, psum[S][L][Hkv][cap] float64 or None)."""
    K, V, q = _c(K), _c(V), _c(q)
    dt = _dt(K)
    assert _dt(V) == dt and _dt(q) == dt
    S, L, Hkv, cap, D = K.shape
    Hq = q.shape[2]
    assert q.shape == (S, L, Hq, D)
    n = np.ascontiguousarray(np.broadcast_to(np.asarray(n, dtype=np.int32), (S,)))
    assert (n >= 0).all() and (n <= cap).all()
    P = plen = 0
    if prefix_K is not None:
        prefix_K, prefix_V = _c(prefix_K), _c(prefix_V)
        assert _dt(prefix_K) == dt and _dt(prefix_V) == dt
        P, _, _, plen, _ = prefix_K.shape
        assert prefix_K.shape == (P, L, Hkv, plen, D) and prefix_V.shape == prefix_K.shape
    out = np.zeros((S, L, Hq, D), np.float64)
    psum = np.zeros((S, L, Hkv, cap), np.float64) if want_psum else None
    rc = lib().orc_decode_attn(_p(K), _p(V), dt, S, L, Hkv, cap, D, _p(prefix_K),
                               _p(prefix_V), P, plen, _p(n), _p(q), Hq, float(scale),
                               _p(out), _p(psum))
    _check(rc, "decode_attn")
    return out, psum


def window_scores(K, V, n, q_win, scale):
    """Importance scores recomputed from the last nq queries q_win[S][L][Hq][nq][D]
    (causal): returns scores[S][L][Hkv][cap] float64."""
    K, V, q_win = _c(K), _c(V), _c(q_win)
    dt = _dt(K)
    S, L, Hkv, cap, D = K.shape
    Hq, nq = q_win.shape[2], q_win.shape[3]
    assert q_win.shape == (S, L, Hq, nq, D)
    n = np.ascontiguousarray(np.broadcast_to(np.asarray(n, dtype=np.int32), (S,)))
    assert (n >= 0).all() and (n <= cap).all()
    scores = np.zeros((S, L, Hkv, cap), np.float64)
    rc = lib().orc_window_scores(_p(K), _p(V), dt, S, L, Hkv, cap, D, _p(n), _p(q_win), Hq,
                                 nq, float(scale), _p(scores))
    _check(rc, "window_scores")
    return scores


def select_topb(score, n, B, W):
    """Kept slot ids (ascending, length B) for one head with n live entries."""
    score = np.ascontiguousarray(np.asarray(score, dtype=np.float64)[:n])
    kept = np.zeros(B, np.int32)
    rc = lib().orc_select_topb(_p(score), int(n), int(B), int(W), _p(kept))
    _check(rc, "select_topb")
    return kept


def compact_head(K, V, pos, kept):
    """In-place compaction of one head: K,V[cap][D] (numpy, contiguous), pos[cap]."""
    assert K.flags.c_contiguous and V.flags.c_contiguous
    dt = _dt(K)
    kept = np.ascontiguousarray(kept, dtype=np.int32)
    rc = lib().orc_compact_head(_p(K), _p(V), _p(pos), dt, K.shape[-1], _p(kept), len(kept))
    _check(rc, "compact_head")


def entropy(logits, V=None, inv_temp=1.0):
    """H[R] float64 of softmax(inv_temp * logits[:, :V])."""
    logits = _c(logits)
    if logits.ndim == 1:
        logits = logits[None]
    R, ld = logits.shape
    V = ld if V is None else V
    H = np.zeros(R, np.float64)
    rc = lib().orc_entropy(_p(logits), _dt(logits), R, int(V), int(ld), float(inv_temp), _p(H))
    _check(rc, "entropy")
    return H


class Detector:
    """Online entropy detector state for R candidates (Eq. (4) moving average)."""

    def __init__(self, R, window=12, guard=24, tau=7.0):
        self.window, self.guard, self.tau = window, guard, tau
        self.hist = np.zeros((R, window), np.float64)
        self.cnt = np.zeros(R, np.int32)
        self.flag = np.zeros(R, np.uint8)

    def step(self, H):
        H = np.ascontiguousarray(H, dtype=np.float64)
        rc = lib().orc_detector_step(_p(H), len(H), _p(self.hist), _p(self.cnt),
                                     _p(self.flag), self.window, self.guard, float(self.tau))
        _check(rc, "detector_step")
        return self.flag.copy()
