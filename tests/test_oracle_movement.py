"""Pins of the fork / commit oracle (oracle/movement.py) against properties
that do not restate its code:

  M1  a fork by a permutation followed by a fork by its inverse restores the
      source exactly;
  M2  slots at or beyond `length`, and destinations with index -1, are left
      bit for bit as they were;
  M3  in-place fan-out (source rows map to themselves) gives N identical
      candidates of each source;
  M4  forking commutes with eviction: evicting N forks of a state equals
      forking the evicted state (each head selects from its own scores);
  M5  one bulk append of T tokens equals T appends of one token;
  M6  a one-pass commit of T >= W tokens that ends exactly at B + buffer + 1
      keeps the same slots, positions and rows as T token-by-token steps of
      the streamed decode loop (oracle/run.py), whose window scores come
      from the per-step attention rows instead of a recomputation;
  M7  a commit that does not overflow B + buffer only appends;
  M8  after an overflowing commit exactly B slots remain, in temporal order,
      and the W newest tokens are among them.
"""
import numpy as np
import pytest

import oracle
from oracle import movement
from oracle.run import BaseOracle

S, L, Hkv, Hq, D = 3, 2, 2, 4, 8
B, W, BUF = 8, 3, 4
CAP = B + BUF + 1


def _state(rng, S_=S, cap=CAP, scores=True):
    st = dict(K=rng.standard_normal((S_, L, Hkv, cap, D)).astype(np.float32),
              V=rng.standard_normal((S_, L, Hkv, cap, D)).astype(np.float32),
              pos=rng.integers(0, 1000, (S_, L, Hkv, cap)).astype(np.int32))
    st["score"] = rng.random((S_, L, Hkv, cap)) if scores else None
    return st


def _copy(st):
    return {k: (None if v is None else v.copy()) for k, v in st.items()}


def _eq(a, b):
    return all((a[k] is None and b[k] is None) or np.array_equal(a[k], b[k]) for k in a)


def test_m1_permutation_round_trip():
    rng = np.random.default_rng(1)
    src = _state(rng, S_=5)
    perm = rng.permutation(5)
    mid = _state(rng, S_=5)
    movement.fork(src, mid, perm, [CAP] * 5)
    back = _state(rng, S_=5)
    movement.fork(mid, back, np.argsort(perm), [CAP] * 5)
    assert _eq(back, src)
    assert not _eq(mid, src)


def test_m2_untouched_slots_and_rows():
    rng = np.random.default_rng(2)
    src, dst = _state(rng), _state(rng)
    before = _copy(dst)
    length = [0, 5, CAP]
    movement.fork(src, dst, [2, -1, 0], length)
    # row 0: length 0 -> untouched; row 1: index -1 -> untouched
    for k in dst:
        assert np.array_equal(dst[k][0], before[k][0])
        assert np.array_equal(dst[k][1], before[k][1])
    # row 2 copied completely from source 0
    for k in dst:
        assert np.array_equal(dst[k][2], src[k][0])
    # a partial copy keeps the tail
    dst2 = _copy(before)
    movement.fork(src, dst2, [-1, -1, 1], [0, 0, 5])
    for k in dst2:
        assert np.array_equal(dst2[k][2, :, :, 5:], before[k][2, :, :, 5:])
        assert not np.array_equal(dst2[k][2, :, :, :5], before[k][2, :, :, :5])


def test_m3_in_place_fan_out():
    rng = np.random.default_rng(3)
    N = 3
    st = _state(rng, S_=2 * N)
    orig = _copy(st)
    idx = [0, 0, 0, 3, 3, 3]
    movement.fork(st, st, idx, [7] * 6)
    for s in range(6):
        r = idx[s]
        for k in st:
            assert np.array_equal(st[k][s, :, :, :7], orig[k][r, :, :, :7])
            assert np.array_equal(st[k][s, :, :, 7:], orig[k][s, :, :, 7:])


def _evict_all(st, n):
    for s in range(st["K"].shape[0]):
        for l in range(L):
            for h in range(Hkv):
                kept = oracle.select_topb(st["score"][s, l, h], n, B, W)
                oracle.compact_head(st["K"][s, l, h], st["V"][s, l, h], st["pos"][s, l, h], kept)


def test_m4_fork_commutes_with_eviction():
    rng = np.random.default_rng(4)
    N = 4
    state = _state(rng, S_=1)
    n = CAP
    a = _state(rng, S_=N)
    movement.fork(state, a, [0] * N, [n] * N)
    _evict_all(a, n)
    ev = _copy(state)
    _evict_all(ev, n)
    b = _state(rng, S_=N)
    movement.fork(ev, b, [0] * N, [B] * N)
    for k in ("K", "V", "pos"):
        assert np.array_equal(a[k][..., :B, :] if a[k].ndim == 5 else a[k][..., :B],
                              b[k][..., :B, :] if b[k].ndim == 5 else b[k][..., :B])


def test_m5_bulk_append_equals_single_appends():
    rng = np.random.default_rng(5)
    T = 6
    c1, c2 = _state(rng, scores=False), None
    c2 = _copy(c1)
    n0 = [0, 3, CAP - T]
    kn = rng.standard_normal((S, L, Hkv, T, D)).astype(np.float32)
    vn = rng.standard_normal((S, L, Hkv, T, D)).astype(np.float32)
    pn = rng.integers(0, 10 ** 6, (S, T)).astype(np.int32)
    movement.append(c1, n0, kn, vn, pn)
    for i in range(T):
        movement.append(c2, [x + i for x in n0], kn[:, :, :, i:i + 1], vn[:, :, :, i:i + 1],
                        pn[:, i:i + 1])
    assert _eq(c1, c2)


def _tokens(rng, T):
    return (rng.standard_normal((S, L, Hq, T, D)).astype(np.float32),
            rng.standard_normal((S, L, Hkv, T, D)).astype(np.float32),
            rng.standard_normal((S, L, Hkv, T, D)).astype(np.float32))


@pytest.mark.parametrize("T", [W, W + 2, BUF + 2])
def test_m6_commit_matches_streamed_decode(T):
    rng = np.random.default_rng(60 + T)
    scale = 0.5
    n0 = B + BUF + 1 - T
    # Prefix of n0 tokens, no eviction on the way (n0 <= B + buffer).
    qp, kp, vp = _tokens(rng, n0)
    q, k, v = _tokens(rng, T)
    ref = BaseOracle(S, L, Hkv, Hq, D, B, W, BUF, np.float32, scale)
    for t in range(n0):
        ref.step(t, qp[:, :, :, t], kp[:, :, :, t], vp[:, :, :, t])
    cache = dict(K=ref.K.copy(), V=ref.V.copy(), pos=ref.pos.copy())
    for i in range(T):
        ref.step(n0 + i, q[:, :, :, i], k[:, :, :, i], v[:, :, :, i])
    assert len(ref.events) == 1
    ev = ref.events[0]
    pos_new = np.tile(np.arange(n0, n0 + T, dtype=np.int32), (S, 1))
    n, score, kept = movement.commit(cache, n0, k, v, pos_new, q, scale, B, W, BUF)
    assert n == B
    np.testing.assert_allclose(score[..., :B + BUF + 1], ev["score"], rtol=0, atol=1e-12)
    assert np.array_equal(kept, ev["kept"])
    assert np.array_equal(cache["K"][..., :B, :], ref.K[..., :B, :])
    assert np.array_equal(cache["V"][..., :B, :], ref.V[..., :B, :])
    assert np.array_equal(cache["pos"][..., :B], ref.pos[..., :B])


def test_m7_commit_without_overflow_only_appends():
    rng = np.random.default_rng(7)
    T = 4
    st = _state(rng, scores=False)
    plain = _copy(st)
    q, k, v = _tokens(rng, T)
    pn = np.tile(np.arange(5, 5 + T, dtype=np.int32), (S, 1))
    n, score, kept = movement.commit(st, 5, k, v, pn, q, 0.3, B, W, BUF)
    movement.append(plain, [5] * S, k, v, pn)
    assert n == 5 + T and kept is None
    assert _eq(st, plain)
    # the recomputed window rows hold probability mass: per query row and
    # query head it sums to 1, so the total is G * min(W, T) per KV head
    np.testing.assert_allclose(score.sum(axis=3), (Hq // Hkv) * min(W, T), rtol=1e-12)


def test_m8_commit_keeps_b_in_order_with_recent_window():
    rng = np.random.default_rng(8)
    T = 11
    n0 = 6
    st = dict(K=np.zeros((S, L, Hkv, n0 + T, D), np.float32),
              V=np.zeros((S, L, Hkv, n0 + T, D), np.float32),
              pos=np.full((S, L, Hkv, n0 + T), -1, np.int32))
    _, kp, vp = _tokens(rng, n0)
    movement.append(st, [0] * S, kp, vp, np.tile(np.arange(n0, dtype=np.int32), (S, 1)))
    q, k, v = _tokens(rng, T)
    movement.commit(st, n0, k, v, np.tile(np.arange(n0, n0 + T, dtype=np.int32), (S, 1)),
                    q, 0.4, B, W, BUF)
    p = st["pos"][..., :B]
    assert np.all(np.diff(p, axis=-1) > 0)
    assert np.all(p[..., B - W:] == np.arange(n0 + T - W, n0 + T))
