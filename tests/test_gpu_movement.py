"""GPU parity of the fork / commit data movement (kvr_fork, kvr_append, and a
one-pass commit = kvr_append + kvr_accumulate_scores + kvr_evict_topb)
against oracle/movement.py, through the C ABI.

Copies are compared bit for bit, including every slot and row the call must
leave untouched (pre-filled with sentinels). The commit's kept sets are
bit-exact wherever the TopB boundary gap of the oracle's fp64 scores is at
least 1e-3, and always equal to the oracle's selection on the GPU's own
float32 scores; its scores are within 1e-4 absolute.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import host, say
from oracle import movement

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_15797_amd import kvr  # noqa: F401  (fails loudly if libkvr.so is missing)
    yield


def kvr():
    from paper_2608_15797_amd import kvr as k
    return k


def _cache(S, L, Hkv, cap, D, dtype, g, pos=True):
    k = kvr()
    K = (torch.randn((S, L, Hkv, cap, D), generator=g)).to(dtype)
    V = (torch.randn((S, L, Hkv, cap, D), generator=g)).to(dtype)
    P = torch.randint(0, 1 << 20, (S, L, Hkv, cap), generator=g, dtype=torch.int32) if pos else None
    return k.Cache(K.to(DEV), V.to(DEV), None if P is None else P.to(DEV))


def _np_state(c, scores=None):
    return dict(K=host(c.k), V=host(c.v), pos=None if c.pos is None else c.pos.cpu().numpy(),
                score=None if scores is None else scores.cpu().numpy())


def _assert_state_equal(got, ref):
    for key in ("K", "V", "pos", "score"):
        if ref.get(key) is None:
            continue
        assert np.array_equal(got[key], ref[key]), key


@pytest.mark.parametrize("dtype,D", [(torch.bfloat16, 128), (torch.float32, 64),
                                     (torch.bfloat16, 64), (torch.float32, 128)])
def test_fork_parity(dtype, D):
    """Fan-out, skipped destinations (-1 and out of range), zero and clamped
    lengths, different caps; K, V, pos and scores."""
    g = torch.Generator().manual_seed(11 + D)
    L, Hkv = 3, 2
    src = _cache(3, L, Hkv, 40, D, dtype, g)
    dst = _cache(9, L, Hkv, 33, D, dtype, g)
    ssc = torch.rand((3, L, Hkv, 40), generator=g).to(DEV)
    dsc = torch.rand((9, L, Hkv, 33), generator=g).to(DEV)
    idx = [0, 0, 0, 1, 1, 2, -1, 5, 2]
    ln = [0, 1, 17, 33, 40, 5, 9, 9, 32]
    ref_src = _np_state(src, ssc)
    ref = _np_state(dst, dsc)
    oidx = [i if 0 <= i < 3 else -1 for i in idx]
    oln = [max(0, min(n, 33)) for n in ln]
    movement.fork(ref_src, ref, oidx, oln)
    kvr().fork(src, dst, torch.tensor(idx, dtype=torch.int32, device=DEV),
               torch.tensor(ln, dtype=torch.int32, device=DEV), ssc, dsc)
    torch.cuda.synchronize()
    _assert_state_equal(_np_state(dst, dsc), ref)
    _assert_state_equal(_np_state(src, ssc), ref_src)  # source untouched


@pytest.mark.parametrize("dtype,D", [(torch.bfloat16, 128), (torch.float32, 64),
                                     (torch.bfloat16, 64), (torch.float32, 128)])
def test_fork_parity_across_pieces(dtype, D):
    """Runs longer than a workgroup's piece of the slots (512 16-byte vectors:
    16 to 64 slots by dtype and D), lengths on every side of the piece
    boundaries, two destination groups of 8 (the second partial), a source
    shared across the group boundary."""
    g = torch.Generator().manual_seed(23 + D)
    L, Hkv = 2, 3
    piece = 512 * 16 // (D * torch.tensor([], dtype=dtype).element_size())
    src = _cache(4, L, Hkv, 300, D, dtype, g)
    dst = _cache(13, L, Hkv, 257, D, dtype, g)
    ssc = torch.rand((4, L, Hkv, 300), generator=g).to(DEV)
    dsc = torch.rand((13, L, Hkv, 257), generator=g).to(DEV)
    idx = [0, 0, 1, 1, 1, 2, 3, 3, 3, 3, 0, 2, -1]
    ln = [piece - 1, piece, piece + 1, 2 * piece + 3, 257, 300, 1, 0, 3 * piece, 4 * piece - 1,
          5 * piece + 7, 100, 50]
    ref_src = _np_state(src, ssc)
    ref = _np_state(dst, dsc)
    oln = [max(0, min(n, 257)) for n in ln]
    movement.fork(ref_src, ref, idx, oln)
    kvr().fork(src, dst, torch.tensor(idx, dtype=torch.int32, device=DEV),
               torch.tensor(ln, dtype=torch.int32, device=DEV), ssc, dsc)
    torch.cuda.synchronize()
    _assert_state_equal(_np_state(dst, dsc), ref)
    _assert_state_equal(_np_state(src, ssc), ref_src)


def test_fork_without_pos_and_scores():
    g = torch.Generator().manual_seed(5)
    src = _cache(2, 2, 2, 24, 128, torch.bfloat16, g)
    dst = _cache(4, 2, 2, 24, 128, torch.bfloat16, g, pos=False)
    ref = _np_state(dst)
    movement.fork(_np_state(src), ref, [1, 0, 1, 0], [24, 3, 0, 11])
    kvr().fork(src, dst, torch.tensor([1, 0, 1, 0], dtype=torch.int32, device=DEV),
               torch.tensor([24, 3, 0, 11], dtype=torch.int32, device=DEV))
    torch.cuda.synchronize()
    _assert_state_equal(_np_state(dst), ref)


def test_fork_in_place_fan_out():
    """Candidate 2 of problem 0 and candidate 0 of problem 1 are retained and
    forked to their siblings inside one cache (sources map to themselves)."""
    g = torch.Generator().manual_seed(6)
    N = 4
    c = _cache(2 * N, 2, 2, 48, 128, torch.bfloat16, g)
    sc = torch.rand((2 * N, 2, 2, 48), generator=g).to(DEV)
    idx = [2, 2, 2, 2, 4, 4, 4, 4]
    ln = [30] * 4 + [48] * 4
    ref = _np_state(c, sc)
    movement.fork(ref, ref, idx, ln)
    kvr().fork(c, c, torch.tensor(idx, dtype=torch.int32, device=DEV),
               torch.tensor(ln, dtype=torch.int32, device=DEV), sc, sc)
    torch.cuda.synchronize()
    _assert_state_equal(_np_state(c, sc), ref)


def test_fork_rejects_bad_arguments():
    k = kvr()
    g = torch.Generator().manual_seed(7)
    a = _cache(2, 2, 2, 16, 128, torch.bfloat16, g)
    b = _cache(2, 3, 2, 16, 128, torch.bfloat16, g)
    nopos = _cache(2, 2, 2, 16, 128, torch.bfloat16, g, pos=False)
    i2 = torch.zeros(2, dtype=torch.int32, device=DEV)
    with pytest.raises(k.KvrError):
        k.fork(a, b, i2, i2)                      # L differs
    with pytest.raises(k.KvrError):
        k.fork(nopos, a, i2, i2)                  # dst tracks pos, src does not
    sc = torch.zeros((2, 2, 2, 16), device=DEV)
    with pytest.raises(k.KvrError):
        k.fork(a, a, i2, i2, sc, None)            # one score pointer


def test_fork_full_shape_sampled():
    """7B shape: 16 trajectory states (cap 641, B + buffer live slots) fanned
    out to 16 x 8 candidates; sampled destinations checked bit for bit."""
    g = torch.Generator(device=DEV).manual_seed(8)
    P, N, L, Hkv, D = 16, 8, 28, 4, 128
    cap = 641
    src = kvr().Cache(torch.randn((P, L, Hkv, cap, D), generator=g, device=DEV).to(torch.bfloat16),
                      torch.randn((P, L, Hkv, cap, D), generator=g, device=DEV).to(torch.bfloat16),
                      torch.randint(0, 1 << 20, (P, L, Hkv, cap), generator=g, device=DEV,
                                    dtype=torch.int32))
    dst = kvr().Cache.empty(P * N, L, Hkv, cap, D, torch.bfloat16)
    dst.k.fill_(7.0)
    dst.v.fill_(-7.0)
    idx = torch.arange(P * N, device=DEV, dtype=torch.int32) // N
    ln = torch.full((P * N,), 640, dtype=torch.int32, device=DEV)
    kvr().fork(src, dst, idx, ln)
    torch.cuda.synchronize()
    for s in (0, 7, 8, 61, 127):
        r = s // N
        assert torch.equal(dst.k[s, :, :, :640], src.k[r, :, :, :640]), s
        assert torch.equal(dst.v[s, :, :, :640], src.v[r, :, :, :640]), s
        assert torch.equal(dst.pos[s, :, :, :640], src.pos[r, :, :, :640]), s
        assert bool((dst.k[s, :, :, 640:] == 7.0).all()) and bool((dst.v[s, :, :, 640:] == -7.0).all())
        assert bool((dst.pos[s, :, :, 640:] == -1).all())


@pytest.mark.parametrize("dtype,D", [(torch.bfloat16, 128), (torch.float32, 64)])
@pytest.mark.parametrize("T", [0, 1, 7, 40])
def test_append_parity(dtype, D, T):
    """Bulk append at lengths 0, mid, exactly cap - T and overflowing the cap
    (rows that do not fit are dropped); untouched slots stay as they were."""
    g = torch.Generator().manual_seed(100 + T + D)
    S, L, Hkv, cap = 4, 2, 3, 48
    c = _cache(S, L, Hkv, cap, D, dtype, g)
    kn = torch.randn((S, L, Hkv, T, D), generator=g).to(dtype)
    vn = torch.randn((S, L, Hkv, T, D), generator=g).to(dtype)
    pn = torch.randint(0, 1 << 20, (S, T), generator=g, dtype=torch.int32)
    ln = [0, 5, cap - T, cap - T // 2 if T else cap]
    ref = _np_state(c)
    for s in range(S):
        fit = max(0, min(T, cap - ln[s]))
        movement.append({k: v[s:s + 1] for k, v in ref.items() if v is not None}, [ln[s]],
                        host(kn[s:s + 1, :, :, :fit]), host(vn[s:s + 1, :, :, :fit]),
                        pn[s:s + 1, :fit].numpy())
    kvr().append(c, torch.tensor(ln, dtype=torch.int32, device=DEV), kn.to(DEV), vn.to(DEV),
                 pn.to(DEV))
    torch.cuda.synchronize()
    _assert_state_equal(_np_state(c), ref)


def test_append_rejects_bad_arguments():
    k = kvr()
    g = torch.Generator().manual_seed(9)
    c = _cache(2, 2, 2, 16, 128, torch.bfloat16, g, pos=False)
    kn = torch.zeros((2, 2, 2, 3, 128), dtype=torch.bfloat16, device=DEV)
    ln = torch.zeros(2, dtype=torch.int32, device=DEV)
    with pytest.raises(k.KvrError):
        k.append(c, ln, kn, kn, torch.zeros((2, 3), dtype=torch.int32, device=DEV))


def _commit_gpu(c, n0, kn, vn, pn, q, scale, B, W, buffer, scores):
    k = kvr()
    S = c.k.shape[0]
    T = kn.shape[3]
    k.append(c, torch.full((S,), n0, dtype=torch.int32, device=DEV), kn, vn, pn)
    n = n0 + T
    nq = min(W, T)
    ln = torch.full((S,), n, dtype=torch.int32, device=DEV)
    k.accumulate_scores(c, ln, q[:, :, :, T - nq:].contiguous(), scale, scores)
    got_scores = scores.cpu().double().numpy()
    kept = None
    if n > B + buffer:
        kept = torch.zeros(c.k.shape[:3] + (B,), dtype=torch.int32, device=DEV)
        k.evict_topb(c, ln, scores, k.Policy(B, W, buffer), kept)
    torch.cuda.synchronize()
    return got_scores, kept


@pytest.mark.parametrize("dtype,D,n0,T", [
    (torch.float32, 64, 10, 24),       # overflow, T > W
    (torch.bfloat16, 128, 20, 17),     # overflow by a few slots
    (torch.bfloat16, 128, 0, 64),      # one-shot prompt compression
    (torch.bfloat16, 128, 22, 5),      # T < W: window of T queries, overflow
    (torch.bfloat16, 64, 3, 9),        # no overflow: append only
])
def test_commit_parity(dtype, D, n0, T):
    g = torch.Generator().manual_seed(1000 + n0 + T)
    S, L, Hkv, G = 3, 2, 2, 4
    B, W, buffer = 16, 8, 8
    cap = max(n0 + T, B + buffer + 1)
    c = _cache(S, L, Hkv, cap, D, dtype, g)
    kn = torch.randn((S, L, Hkv, T, D), generator=g).to(dtype)
    vn = torch.randn((S, L, Hkv, T, D), generator=g).to(dtype)
    q = torch.randn((S, L, Hkv * G, T, D), generator=g).to(dtype)
    pn = (torch.arange(n0, n0 + T, dtype=torch.int32)).repeat(S, 1)
    scale = D ** -0.5
    ref = _np_state(c)
    pre = dict(K=ref["K"].copy(), V=ref["V"].copy(), pos=ref["pos"].copy())
    movement.append(pre, [n0] * S, host(kn), host(vn), pn.numpy())
    n_ref, sc_ref, kept_ref = movement.commit(ref, n0, host(kn), host(vn), pn.numpy(), host(q),
                                              scale, B, W, buffer)
    scores = torch.zeros((S, L, Hkv, cap), device=DEV)
    got_sc, kept = _commit_gpu(c, n0, kn.to(DEV), vn.to(DEV), pn.to(DEV), q.to(DEV), scale,
                               B, W, buffer, scores)
    n = n0 + T
    d = np.abs(got_sc[..., :n] - sc_ref[..., :n]).max()
    say("commit n0=%d T=%d: score max abs err %.2e" % (n0, T, d))
    assert d <= 1e-4
    got = _np_state(c)
    if kept_ref is None:
        assert kept is None
        _assert_state_equal(got, ref)
        return
    kept = kept.cpu().numpy()
    near = 0
    for idx in np.ndindex(*kept.shape[:3]):
        assert np.array_equal(oracle.select_topb(got_sc[idx], n, B, W), kept[idx]), idx
        cands = np.sort(sc_ref[idx][: n - W])[::-1]
        if cands[B - W - 1] - cands[B - W] >= 1e-3:
            assert np.array_equal(kept[idx], kept_ref[idx]), idx
        else:
            near += 1
        src = kept[idx]
        assert np.array_equal(got["K"][idx][:B], pre["K"][idx][src])
        assert np.array_equal(got["V"][idx][:B], pre["V"][idx][src])
        assert np.array_equal(got["pos"][idx][:B], pre["pos"][idx][src])
    say("  near ties (gap < 1e-3): %d of %d heads" % (near, kept.shape[0] * kept.shape[1] * kept.shape[2]))
