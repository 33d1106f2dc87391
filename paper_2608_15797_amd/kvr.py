"""Python binding of libkvr (ctypes). Argument marshalling only.

Every function takes torch tensors that already live on the GPU, passes their
device pointers and sizes to the C ABI declared in include/kvr.h, and raises
KvrError on a non-zero status. All computation happens in the HIP kernels;
there is no fallback: if libkvr.so is missing, importing this module fails.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkvr.so")

KVR_F32, KVR_BF16 = 0, 1
STATUS = {0: "KVR_OK", -1: "KVR_EINVAL", -2: "KVR_EUNSUPPORTED", -3: "KVR_EHIP",
          -4: "KVR_EWORKSPACE"}

# Every symbol declared in include/kvr.h.
EXPORTS = ("kvr_strerror", "kvr_last_error", "kvr_decode_attn", "kvr_decode_attn_workspace_size",
           "kvr_accumulate_scores", "kvr_evict_topb", "kvr_logit_entropy",
           "kvr_logit_entropy_workspace_size", "kvr_fork", "kvr_append",
           "kvr_logit_entropy_sample", "kvr_logit_entropy_sample_workspace_size",
           "kvr_redundancy_scores", "kvr_logit_entropy_batch", "kvr_logit_entropy_batch_workspace_size",
           "kvr_logit_entropy_batch_noalloc", "kvr_decode_attn_entropy", "kvr_decode_attn_entropy_sample")


class KvrError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__("%s failed: %s (%s)" % (where, STATUS.get(status, status), detail))
        self.status = status


class c_cache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("pos", ctypes.c_void_p),
                ("S", ctypes.c_int32), ("L", ctypes.c_int32), ("Hkv", ctypes.c_int32),
                ("cap", ctypes.c_int32), ("D", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class c_prefix(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("P", ctypes.c_int32),
                ("plen", ctypes.c_int32)]


class c_policy(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("W", ctypes.c_int32), ("buffer", ctypes.c_int32)]


class c_detector(ctypes.Structure):
    _fields_ = [("hist", ctypes.c_void_p), ("cnt", ctypes.c_void_p), ("flag", ctypes.c_void_p),
                ("window", ctypes.c_int32), ("guard", ctypes.c_int32), ("tau", ctypes.c_float)]


class c_logit_set(ctypes.Structure):
    _fields_ = [("logits", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("R", ctypes.c_int32),
                ("V", ctypes.c_int32), ("ld", ctypes.c_int64), ("inv_temp", ctypes.c_float),
                ("H", ctypes.c_void_p), ("det", ctypes.POINTER(c_detector))]


class c_sampler(ctypes.Structure):
    _fields_ = [("temperature", ctypes.c_float), ("top_k", ctypes.c_int32), ("top_p", ctypes.c_float),
                ("seed", ctypes.c_uint64), ("step", ctypes.c_uint64)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError("libkvr.so not built: run `python -m paper_2608_15797_amd.build` "
                          "(or __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, f32, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                             ctypes.c_size_t)
    P = ctypes.POINTER
    lib.kvr_strerror.argtypes = [ctypes.c_int]
    lib.kvr_strerror.restype = ctypes.c_char_p
    lib.kvr_last_error.argtypes = []
    lib.kvr_last_error.restype = ctypes.c_char_p
    lib.kvr_decode_attn.argtypes = [P(c_cache), P(c_prefix), vp, vp, i32, f32, vp, vp, vp, vp,
                                    P(c_policy), vp, vp, sz, vp]
    lib.kvr_decode_attn.restype = ctypes.c_int
    lib.kvr_decode_attn_workspace_size.argtypes = [P(c_cache), P(c_prefix), i32]
    lib.kvr_decode_attn_workspace_size.restype = sz
    lib.kvr_accumulate_scores.argtypes = [P(c_cache), vp, vp, i32, i32, f32, vp, i32, vp]
    lib.kvr_accumulate_scores.restype = ctypes.c_int
    lib.kvr_evict_topb.argtypes = [P(c_cache), vp, vp, vp, P(c_policy), vp, vp]
    lib.kvr_evict_topb.restype = ctypes.c_int
    lib.kvr_logit_entropy.argtypes = [vp, i32, i32, i32, i64, f32, vp, P(c_detector), vp, sz, vp]
    lib.kvr_logit_entropy.restype = ctypes.c_int
    lib.kvr_logit_entropy_workspace_size.argtypes = [i32, i32]
    lib.kvr_logit_entropy_workspace_size.restype = sz
    lib.kvr_logit_entropy_batch.argtypes = [P(c_logit_set), i32, vp, sz, vp]
    lib.kvr_logit_entropy_batch.restype = ctypes.c_int
    lib.kvr_logit_entropy_batch_workspace_size.argtypes = [P(c_logit_set), i32]
    lib.kvr_logit_entropy_batch_workspace_size.restype = sz
    lib.kvr_decode_attn_entropy.argtypes = [P(c_cache), P(c_prefix), vp, vp, i32, f32, vp, vp, vp, vp,
                                            P(c_policy), vp, vp, sz, P(c_logit_set), i32, vp]
    lib.kvr_decode_attn_entropy.restype = ctypes.c_int
    lib.kvr_decode_attn_entropy_sample.argtypes = [P(c_cache), P(c_prefix), vp, vp, i32, f32, vp, vp, vp, vp,
                                                   P(c_policy), vp, vp, sz, P(c_logit_set), i32, P(c_sampler),
                                                   P(vp), vp]
    lib.kvr_decode_attn_entropy_sample.restype = ctypes.c_int
    lib.kvr_logit_entropy_batch_noalloc.argtypes = [P(c_logit_set), i32, vp]
    lib.kvr_logit_entropy_batch_noalloc.restype = ctypes.c_int
    lib.kvr_logit_entropy_sample.argtypes = [vp, i32, i32, i32, i64, f32, vp, P(c_detector),
                                             P(c_sampler), vp, vp, sz, vp]
    lib.kvr_logit_entropy_sample.restype = ctypes.c_int
    lib.kvr_logit_entropy_sample_workspace_size.argtypes = [i32, i32, i32]
    lib.kvr_logit_entropy_sample_workspace_size.restype = sz
    lib.kvr_redundancy_scores.argtypes = [P(c_cache), vp, vp, P(c_policy), f32, i32, vp, vp]
    lib.kvr_redundancy_scores.restype = ctypes.c_int
    lib.kvr_fork.argtypes = [P(c_cache), P(c_cache), vp, vp, vp, vp, vp]
    lib.kvr_fork.restype = ctypes.c_int
    lib.kvr_append.argtypes = [P(c_cache), vp, i32, vp, vp, vp, vp]
    lib.kvr_append.restype = ctypes.c_int
    return lib


lib = _load()


def _check(rc: int, where: str):
    if rc != 0:
        raise KvrError(rc, where, (lib.kvr_last_error() or b"").decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def dtype_code(dt: torch.dtype) -> int:
    if dt == torch.float32:
        return KVR_F32
    if dt == torch.bfloat16:
        return KVR_BF16
    raise TypeError("libkvr handles float32 and bfloat16, not %s" % dt)


@dataclass
class Cache:
    """Per-sequence KV cache K,V[S][L][Hkv][cap][D] (+ pos[S][L][Hkv][cap])."""
    k: torch.Tensor
    v: torch.Tensor
    pos: Optional[torch.Tensor] = None

    @staticmethod
    def empty(S, L, Hkv, cap, D, dtype, device="cuda", with_pos=True):
        k = torch.empty((S, L, Hkv, cap, D), dtype=dtype, device=device)
        v = torch.empty_like(k)
        pos = torch.full((S, L, Hkv, cap), -1, dtype=torch.int32, device=device) if with_pos else None
        return Cache(k, v, pos)

    def c(self) -> c_cache:
        cached = self.__dict__.get("_c")
        if cached is not None and cached[0] == (self.k.data_ptr(), self.v.data_ptr(),
                                                None if self.pos is None else self.pos.data_ptr()):
            return cached[1]
        S, L, Hkv, cap, D = self.k.shape
        assert self.k.is_contiguous() and self.v.is_contiguous() and self.v.shape == self.k.shape
        if self.pos is not None:
            assert self.pos.shape == (S, L, Hkv, cap) and self.pos.dtype == torch.int32
        cc = c_cache(self.k.data_ptr(), self.v.data_ptr(),
                     None if self.pos is None else self.pos.data_ptr(),
                     S, L, Hkv, cap, D, dtype_code(self.k.dtype))
        self.__dict__["_c"] = ((self.k.data_ptr(), self.v.data_ptr(),
                                None if self.pos is None else self.pos.data_ptr()), cc)
        return cc


@dataclass
class Prefix:
    """Shared full-context prefix K,V[P][L][Hkv][plen][D]."""
    k: torch.Tensor
    v: torch.Tensor

    def c(self) -> c_prefix:
        assert self.k.is_contiguous() and self.v.is_contiguous()
        return c_prefix(self.k.data_ptr(), self.v.data_ptr(), self.k.shape[0], self.k.shape[3])


@dataclass
class Policy:
    B: int
    W: int
    buffer: int

    def c(self) -> c_policy:
        return c_policy(self.B, self.W, self.buffer)


@dataclass
class Detector:
    """Entropy-detector state for R rows; starts zeroed."""
    hist: torch.Tensor
    cnt: torch.Tensor
    flag: torch.Tensor
    window: int = 12
    guard: int = 24
    tau: float = 7.0

    @staticmethod
    def zeros(R, window=12, guard=24, tau=7.0, device="cuda"):
        return Detector(torch.zeros((R, window), dtype=torch.float32, device=device),
                        torch.zeros(R, dtype=torch.int32, device=device),
                        torch.zeros(R, dtype=torch.uint8, device=device), window, guard, tau)

    def c(self) -> c_detector:
        return c_detector(self.hist.data_ptr(), self.cnt.data_ptr(), self.flag.data_ptr(),
                          self.window, self.guard, self.tau)


def decode_attn_workspace_size(cache: Cache, prefix: Optional[Prefix], Hq: int) -> int:
    cc = cache.c()
    pc = prefix.c() if prefix is not None else None
    return int(lib.kvr_decode_attn_workspace_size(ctypes.byref(cc),
                                                  ctypes.byref(pc) if pc else None, Hq))


def decode_attn(cache: Cache, len_: torch.Tensor, q: torch.Tensor, out: torch.Tensor,
                scale: float, k_new=None, v_new=None, new_pos=None,
                prefix: Optional[Prefix] = None, policy: Optional[Policy] = None,
                scores: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                stream=None) -> None:
    """kvr_decode_attn: q[S][L][Hq][D] -> out, appending k_new/v_new at len-1."""
    cc = cache.c()
    pc = prefix.c() if prefix is not None else None
    pol = policy.c() if policy is not None else None
    for t in (len_, q, out, k_new, v_new, new_pos, scores, workspace):
        assert t is None or t.is_contiguous()
    rc = lib.kvr_decode_attn(ctypes.byref(cc), ctypes.byref(pc) if pc else None, _ptr(len_),
                             _ptr(q), q.shape[2], float(scale), _ptr(k_new), _ptr(v_new),
                             _ptr(new_pos), _ptr(out), ctypes.byref(pol) if pol else None,
                             _ptr(scores), _ptr(workspace),
                             0 if workspace is None else workspace.numel() * workspace.element_size(),
                             _stream(stream))
    _check(rc, "kvr_decode_attn")


def decode_attn_entropy(cache: Cache, len_: torch.Tensor, q: torch.Tensor, out: torch.Tensor, scale: float,
                        sets, k_new=None, v_new=None, new_pos=None, prefix: Optional[Prefix] = None,
                        policy: Optional[Policy] = None, scores: Optional[torch.Tensor] = None,
                        workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """kvr_decode_attn_entropy: decode_attn plus the entropies of the LogitSet
    list `sets` in the same launch (the context launch with a prefix)."""
    cc = cache.c()
    pc = prefix.c() if prefix is not None else None
    pol = policy.c() if policy is not None else None
    for t in (len_, q, out, k_new, v_new, new_pos, scores, workspace):
        assert t is None or t.is_contiguous()
    arr = _logit_sets(sets)
    rc = lib.kvr_decode_attn_entropy(ctypes.byref(cc), ctypes.byref(pc) if pc else None, _ptr(len_), _ptr(q),
                                     q.shape[2], float(scale), _ptr(k_new), _ptr(v_new), _ptr(new_pos), _ptr(out),
                                     ctypes.byref(pol) if pol else None, _ptr(scores), _ptr(workspace),
                                     0 if workspace is None else workspace.numel() * workspace.element_size(),
                                     arr, len(sets), _stream(stream))
    _check(rc, "kvr_decode_attn_entropy")


def decode_attn_entropy_sample(cache: Cache, len_: torch.Tensor, q: torch.Tensor, out: torch.Tensor, scale: float,
                               sets, sampler, tokens, k_new=None, v_new=None, new_pos=None,
                               prefix: Optional[Prefix] = None, policy: Optional[Policy] = None,
                               scores: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                               stream=None) -> None:
    """kvr_decode_attn_entropy_sample: decode_attn_entropy plus the next token
    of every row of every LogitSet; `tokens` holds one int32 tensor per set."""
    cc = cache.c()
    pc = prefix.c() if prefix is not None else None
    pol = policy.c() if policy is not None else None
    for t in (len_, q, out, k_new, v_new, new_pos, scores, workspace, *tokens):
        assert t is None or t.is_contiguous()
    assert len(tokens) == len(sets)
    arr = _logit_sets(sets)
    tp = (ctypes.c_void_p * len(tokens))(*[t.data_ptr() for t in tokens])
    rc = lib.kvr_decode_attn_entropy_sample(ctypes.byref(cc), ctypes.byref(pc) if pc else None, _ptr(len_),
                                            _ptr(q), q.shape[2], float(scale), _ptr(k_new), _ptr(v_new),
                                            _ptr(new_pos), _ptr(out), ctypes.byref(pol) if pol else None,
                                            _ptr(scores), _ptr(workspace),
                                            0 if workspace is None else workspace.numel() * workspace.element_size(),
                                            arr, len(sets), ctypes.byref(sampler.c()), tp, _stream(stream))
    _check(rc, "kvr_decode_attn_entropy_sample")


def accumulate_scores(cache: Cache, len_: torch.Tensor, q_win: torch.Tensor, scale: float,
                      scores: torch.Tensor, accumulate: bool = False, stream=None) -> None:
    """kvr_accumulate_scores: q_win[S][L][Hq][nq][D]."""
    cc = cache.c()
    assert q_win.is_contiguous() and scores.is_contiguous()
    rc = lib.kvr_accumulate_scores(ctypes.byref(cc), _ptr(len_), _ptr(q_win), q_win.shape[3],
                                   q_win.shape[2], float(scale), _ptr(scores), int(accumulate),
                                   _stream(stream))
    _check(rc, "kvr_accumulate_scores")


def evict_topb(cache: Cache, len_: torch.Tensor, scores: torch.Tensor, policy: Policy,
               kept: Optional[torch.Tensor] = None, len_out: Optional[torch.Tensor] = None,
               stream=None) -> None:
    """kvr_evict_topb: in-place compaction of sequences with len > B + buffer;
    len_out (optional) receives the new live lengths."""
    cc = cache.c()
    pol = policy.c()
    rc = lib.kvr_evict_topb(ctypes.byref(cc), _ptr(len_), _ptr(len_out), _ptr(scores), ctypes.byref(pol),
                            _ptr(kept), _stream(stream))
    _check(rc, "kvr_evict_topb")


def logit_entropy_workspace_size(R: int, V: int) -> int:
    return int(lib.kvr_logit_entropy_workspace_size(R, V))


def logit_entropy(logits: torch.Tensor, H: torch.Tensor, V: Optional[int] = None,
                  inv_temp: float = 1.0, detector: Optional[Detector] = None,
                  workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """kvr_logit_entropy over logits[R][ld] (first V columns)."""
    assert logits.dim() == 2 and logits.stride(1) == 1
    R, ld = logits.shape[0], logits.stride(0)
    V = logits.shape[1] if V is None else V
    det = detector.c() if detector is not None else None
    rc = lib.kvr_logit_entropy(_ptr(logits), dtype_code(logits.dtype), R, V, ld, float(inv_temp),
                               _ptr(H), ctypes.byref(det) if det else None, _ptr(workspace),
                               0 if workspace is None else workspace.numel() * workspace.element_size(),
                               _stream(stream))
    _check(rc, "kvr_logit_entropy")


@dataclass
class LogitSet:
    """One set of logit rows of kvr_logit_entropy_batch: logits[R][ld] (first
    V columns), H[R] output, optional detector."""
    logits: torch.Tensor
    H: torch.Tensor
    V: Optional[int] = None
    inv_temp: float = 1.0
    detector: Optional[Detector] = None


def _logit_sets(sets) -> ctypes.Array:
    arr = (c_logit_set * len(sets))()
    for k, s in enumerate(sets):
        lg = s.logits
        assert lg.dim() == 2 and lg.stride(1) == 1
        det = ctypes.pointer(s.detector.c()) if s.detector is not None else None
        arr[k] = c_logit_set(_ptr(lg), dtype_code(lg.dtype), lg.shape[0],
                             lg.shape[1] if s.V is None else s.V, lg.stride(0), float(s.inv_temp),
                             _ptr(s.H), det)
    return arr


def logit_entropy_batch_workspace_size(shapes, dtype=torch.bfloat16) -> int:
    """Workspace bytes of kvr_logit_entropy_batch for sets of (R, V) rows of
    `dtype` (the size depends on the shapes only)."""
    arr = (c_logit_set * len(shapes))()
    for k, (R, V) in enumerate(shapes):
        arr[k] = c_logit_set(None, dtype_code(dtype), R, V, V, 1.0, None, None)
    return int(lib.kvr_logit_entropy_batch_workspace_size(arr, len(shapes)))


def logit_entropy_batch(sets, workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """kvr_logit_entropy_batch over a list of LogitSet (one launch for all rows)."""
    arr = _logit_sets(sets)
    rc = lib.kvr_logit_entropy_batch(arr, len(sets), _ptr(workspace),
                                     0 if workspace is None else workspace.numel() * workspace.element_size(),
                                     _stream(stream))
    _check(rc, "kvr_logit_entropy_batch")


ENTROPY_SCRATCH_BYTES = 1 << 20  # KVR_ENTROPY_SCRATCH_BYTES


def logit_entropy_batch_noalloc(sets, stream=None) -> None:
    """kvr_logit_entropy_batch_noalloc: as logit_entropy_batch, with the split
    partials in the library's own device scratch (no workspace argument)."""
    arr = _logit_sets(sets)
    rc = lib.kvr_logit_entropy_batch_noalloc(arr, len(sets), _stream(stream))
    _check(rc, "kvr_logit_entropy_batch_noalloc")


def fork(src: Cache, dst: Cache, src_index: torch.Tensor, len_: torch.Tensor,
         src_scores: Optional[torch.Tensor] = None, dst_scores: Optional[torch.Tensor] = None,
         stream=None) -> None:
    """kvr_fork: slots [0, len[s]) of sequence src_index[s] of src -> sequence s of dst."""
    sc, dc = src.c(), dst.c()
    for t in (src_index, len_, src_scores, dst_scores):
        assert t is None or (t.is_contiguous() and t.is_cuda)
    rc = lib.kvr_fork(ctypes.byref(sc), ctypes.byref(dc), _ptr(src_index), _ptr(len_),
                      _ptr(src_scores), _ptr(dst_scores), _stream(stream))
    _check(rc, "kvr_fork")


def append(cache: Cache, len_: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
           pos_new: Optional[torch.Tensor] = None, stream=None) -> None:
    """kvr_append: k_new, v_new [S][L][Hkv][T][D] to slots len[s] .. len[s]+T-1."""
    cc = cache.c()
    for t in (len_, k_new, v_new, pos_new):
        assert t is None or t.is_contiguous()
    rc = lib.kvr_append(ctypes.byref(cc), _ptr(len_), k_new.shape[3], _ptr(k_new), _ptr(v_new),
                        _ptr(pos_new), _stream(stream))
    _check(rc, "kvr_append")


@dataclass
class Sampler:
    """Sampling settings of kvr_logit_entropy_sample (decoding setup of the paper:
    temperature 0.8, top-k 20, top-p 0.95)."""
    temperature: float = 0.8
    top_k: int = 20
    top_p: float = 0.95
    seed: int = 0
    step: int = 0

    def c(self) -> c_sampler:
        return c_sampler(self.temperature, self.top_k, self.top_p, self.seed, self.step)


def logit_entropy_sample_workspace_size(R: int, V: int, top_k: int) -> int:
    return int(lib.kvr_logit_entropy_sample_workspace_size(R, V, top_k))


def logit_entropy_sample(logits: torch.Tensor, H: torch.Tensor, tokens: torch.Tensor,
                         sampler: Sampler, V: Optional[int] = None, inv_temp: float = 1.0,
                         detector: Optional[Detector] = None,
                         workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """kvr_logit_entropy_sample: entropy (and detector) plus one sampled token per row."""
    assert logits.dim() == 2 and logits.stride(1) == 1
    R, ld = logits.shape[0], logits.stride(0)
    V = logits.shape[1] if V is None else V
    det = detector.c() if detector is not None else None
    smp = sampler.c()
    rc = lib.kvr_logit_entropy_sample(_ptr(logits), dtype_code(logits.dtype), R, V, ld,
                                      float(inv_temp), _ptr(H), ctypes.byref(det) if det else None,
                                      ctypes.byref(smp), _ptr(tokens), _ptr(workspace),
                                      0 if workspace is None else workspace.numel() * workspace.element_size(),
                                      _stream(stream))
    _check(rc, "kvr_logit_entropy_sample")


def redundancy_scores(cache: Cache, len_: torch.Tensor, importance: torch.Tensor, policy: Policy,
                      out: torch.Tensor, lam: float = 0.1, pool: int = 7, stream=None) -> None:
    """kvr_redundancy_scores: pooled importance mixed with mean key cosine
    similarity, for sequences that evict this step; feed `out` to evict_topb."""
    cc = cache.c()
    pol = policy.c()
    assert importance.is_contiguous() and out.is_contiguous()
    rc = lib.kvr_redundancy_scores(ctypes.byref(cc), _ptr(len_), _ptr(importance), ctypes.byref(pol),
                                   float(lam), int(pool), _ptr(out), _stream(stream))
    _check(rc, "kvr_redundancy_scores")
