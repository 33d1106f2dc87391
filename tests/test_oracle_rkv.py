"""Pins of the redundancy-aware score oracle (oracle/rkv.py).

The composition (how importance and redundancy are normalised and mixed) is a
reading of the paper, which gives no formula, so its parity against the paper
is unpinned. Its pieces and limits are pinned here by facts that do not
restate the oracle's code:

  K1  a regular simplex of m unit keys has every pairwise cosine -1/(m-1), so
      every key's mean cosine is -1/(m-1);
  K2  duplicate keys (any positive scales) have mean cosine 1; in {v, v, -v}
      the mean cosines are 0, 0 and -1;
  K3  sum identity: sum_c R_c = (|sum_c k_c/|k_c||^2 - m) / (m - 1);
  K4  mean cosine is invariant to positive per-key scaling;
  K5  a zero key has cosine 0 with every key;
  K6  max pooling spreads a spike over pool // 2 slots either side, clipped;
  K7  lam = 1 without pooling selects exactly the TopB of the importance
      scores (the pinned selection of the plain evictor);
  K8  lam = 0 keeps keys that are not duplicated before duplicated ones;
  K9  the score sums to 2 lam - 1 over the candidates (both terms are
      normalised to sum to 1).
"""
import numpy as np
import pytest

import oracle
from oracle import rkv


def test_k1_regular_simplex():
    for m in (2, 3, 7, 20):
        D = m + 3
        E = np.zeros((m, D))
        E[:, :m] = np.eye(m) - 1.0 / m
        R = rkv.mean_cosine(E * np.arange(1, m + 1)[:, None])
        np.testing.assert_allclose(R, -1.0 / (m - 1), rtol=0, atol=1e-12)


def test_k2_duplicates_and_antipodes():
    v = np.array([0.3, -1.2, 2.0, 0.5])
    np.testing.assert_allclose(rkv.mean_cosine(np.stack([v, 2 * v, 0.1 * v])), 1.0, atol=1e-12)
    np.testing.assert_allclose(rkv.mean_cosine(np.stack([v, v, -v])), [0.0, 0.0, -1.0], atol=1e-12)


def test_k3_sum_identity():
    rng = np.random.default_rng(3)
    for m, D in ((5, 8), (40, 16), (130, 64)):
        K = rng.standard_normal((m, D)) * rng.uniform(0.1, 3, (m, 1))
        R = rkv.mean_cosine(K)
        U = K / np.linalg.norm(K, axis=1, keepdims=True)
        s = U.sum(axis=0)
        assert abs(R.sum() - (s @ s - m) / (m - 1)) <= 1e-10


def test_k4_scale_invariance():
    rng = np.random.default_rng(4)
    K = rng.standard_normal((30, 16))
    np.testing.assert_allclose(rkv.mean_cosine(K), rkv.mean_cosine(K * rng.uniform(0.01, 50, (30, 1))),
                               rtol=0, atol=1e-12)


def test_k5_zero_key():
    rng = np.random.default_rng(5)
    K = rng.standard_normal((6, 8))
    base = rkv.mean_cosine(K)
    K0 = np.vstack([K, np.zeros((1, 8))])
    R0 = rkv.mean_cosine(K0)
    assert R0[-1] == 0.0
    np.testing.assert_allclose(R0[:-1], base * 5 / 6, atol=1e-12)   # same sums, one more "other"


def test_k6_max_pool():
    I = np.zeros(12)
    I[1] = 5.0
    I[9] = 2.0
    P = rkv.max_pool(I, 7)
    assert list(P) == [5.0, 5.0, 5.0, 5.0, 5.0, 0.0, 2.0, 2.0, 2.0, 2.0, 2.0, 2.0]
    np.testing.assert_array_equal(rkv.max_pool(I, 1), I)


def test_k7_importance_only_limit():
    rng = np.random.default_rng(7)
    B, W, n, D = 16, 4, 40, 8
    K = rng.standard_normal((n, D))
    I = rng.permutation(n).astype(np.float64) * 1e-2 + 0.5
    Z = np.zeros(n)
    Z[: n - W] = rkv.rkv_head(K, I, n, W, 1.0, 1)
    assert np.array_equal(oracle.select_topb(Z, n, B, W), oracle.select_topb(I, n, B, W))


def test_k8_redundancy_only_keeps_unique_keys():
    rng = np.random.default_rng(8)
    B, W, D = 12, 2, 64
    uniq = np.eye(D)[:8] * rng.uniform(0.5, 2, (8, 1))           # mutually orthogonal: R = 0
    dup = np.tile(rng.standard_normal(D), (20, 1)) * rng.uniform(0.5, 2, (20, 1))
    dup[:, :8] = 0.0                                              # orthogonal to the unique keys
    K = np.vstack([dup[:10], uniq, dup[10:], rng.standard_normal((W, D))])
    n = len(K)
    I = rng.uniform(0, 1, n)
    Z = np.zeros(n)
    Z[: n - W] = rkv.rkv_head(K, I, n, W, 0.0, 7)
    kept = oracle.select_topb(Z, n, B, W)
    assert set(range(10, 18)) <= set(kept.tolist())             # all 8 unique keys kept


@pytest.mark.parametrize("lam", [0.0, 0.1, 0.5, 1.0])
def test_k9_normalisation(lam):
    rng = np.random.default_rng(9)
    n, W = 50, 5
    Z = rkv.rkv_head(rng.standard_normal((n, 16)), rng.uniform(0, 3, n), n, W, lam, 7)
    assert abs(Z.sum() - (2 * lam - 1)) <= 1e-12
