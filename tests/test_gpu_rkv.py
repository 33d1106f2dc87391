"""GPU parity of kvr_redundancy_scores (pooled importance mixed with mean key
cosine similarity; oracle/rkv.py) and of eviction driven by it, through the C
ABI.

Scores: within 1e-6 absolute plus 1e-4 relative of the oracle's fp64 values
(the score is O(1/m); float32 sums of m unit vectors). Slots past each head's
candidates and sequences that do not evict are left as they were. Kept sets:
equal to the oracle's TopB on the GPU's own scores bit for bit, and to the
oracle's TopB on its fp64 scores wherever the boundary gap is at least 1e-6.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import host, say
from oracle import rkv

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


CASES = [
    # S, L, Hkv, D, B, W, buffer, dtype, lam, pool
    (3, 2, 2, 128, 32, 8, 24, torch.bfloat16, 0.1, 7),
    (2, 2, 2, 64, 40, 5, 30, torch.bfloat16, 0.5, 3),
    (3, 1, 2, 128, 20, 4, 12, torch.float32, 0.1, 7),
    (2, 1, 3, 64, 16, 8, 16, torch.float32, 1.0, 1),
    (2, 1, 1, 128, 64, 16, 64, torch.bfloat16, 0.0, 7),
    # Heads longer than the keys a lane keeps in registers between the two
    # passes (256 candidates of a float32 D = 128 head, 1024 of a bf16 D = 64
    # head, 512 of a bf16 D = 128 head): the rest is read twice.
    (2, 1, 2, 128, 600, 16, 100, torch.float32, 0.1, 7),
    (2, 1, 2, 64, 1100, 32, 100, torch.bfloat16, 0.1, 5),
    (1, 1, 2, 128, 900, 64, 200, torch.bfloat16, 0.3, 7),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "S%dL%dHkv%dD%d_B%dW%dbuf%d_%s_lam%g_pool%d" % (
    *c[:7], str(c[7]).split(".")[-1], c[8], c[9]))
def test_redundancy_scores_parity(case):
    S, L, Hkv, D, B, W, buffer, dt, lam, pool = case
    k = kvr()
    cap = B + buffer + 1
    g = torch.Generator().manual_seed(cap * 13 + D)
    K = torch.randn((S, L, Hkv, cap, D), generator=g).to(dt)
    K[0, 0, 0, 3] = 0                                  # a zero key
    if cap > 12:
        K[:, :, :, 7] = K[:, :, :, 9] * 2              # duplicated directions
    imp = torch.rand((S, L, Hkv, cap), generator=g)
    imp[:, :, :, 5] = 0
    lens = [cap if s % 2 == 0 else cap - 1 for s in range(S)]   # odd sequences do not evict
    cache = k.Cache(K.to(DEV), K.to(DEV), None)
    out = torch.full((S, L, Hkv, cap), -7.0, device=DEV)
    k.redundancy_scores(cache, torch.tensor(lens, dtype=torch.int32, device=DEV), imp.to(DEV),
                        k.Policy(B, W, buffer), out, lam=lam, pool=pool)
    torch.cuda.synchronize()
    got = out.cpu().double().numpy()
    Kh, Ih = host(K), imp.double().numpy()
    worst = 0.0
    for s in range(S):
        n = lens[s]
        if n <= B + buffer:
            assert (got[s] == -7.0).all()
            continue
        m = n - W
        for l in range(L):
            for h in range(Hkv):
                ref = rkv.rkv_head(Kh[s, l, h], Ih[s, l, h], n, W, lam, pool)
                d = np.abs(got[s, l, h, :m] - ref)
                assert (d <= 1e-6 + 1e-4 * np.abs(ref)).all(), d.max()
                worst = max(worst, d.max())
                assert (got[s, l, h, m:] == -7.0).all()
                assert abs(got[s, l, h, :m].sum() - (2 * lam - 1)) <= 1e-4
    say("  max abs err %.2e" % worst)


def test_redundancy_in_place_then_evict():
    """out aliases the importance array; the scores then drive kvr_evict_topb."""
    k = kvr()
    S, L, Hkv, D, B, W, buffer = 2, 2, 2, 128, 48, 16, 48
    cap = B + buffer + 1
    g = torch.Generator().manual_seed(77)
    K = torch.randn((S, L, Hkv, cap, D), generator=g).to(torch.bfloat16)
    V = torch.randn((S, L, Hkv, cap, D), generator=g).to(torch.bfloat16)
    pos = torch.arange(cap, dtype=torch.int32).repeat(S, L, Hkv, 1)
    imp = torch.rand((S, L, Hkv, cap), generator=g)
    ref = rkv.rkv_scores(host(K), imp.double().numpy(), [cap] * S, W, 0.1, 7)
    cache = k.Cache(K.to(DEV), V.to(DEV), pos.to(DEV))
    sc = imp.to(DEV)
    ln = torch.full((S,), cap, dtype=torch.int32, device=DEV)
    k.redundancy_scores(cache, ln, sc, k.Policy(B, W, buffer), sc, lam=0.1, pool=7)
    got = sc.cpu().double().numpy()
    kept = torch.zeros((S, L, Hkv, B), dtype=torch.int32, device=DEV)
    k.evict_topb(cache, ln, sc, k.Policy(B, W, buffer), kept)
    torch.cuda.synchronize()
    kept = kept.cpu().numpy()
    Kg = host(cache.k)
    checked = 0
    for idx in np.ndindex(S, L, Hkv):
        m = cap - W
        np.testing.assert_allclose(got[idx][:m], ref[idx][:m], rtol=1e-4, atol=1e-6)
        assert np.array_equal(oracle.select_topb(got[idx], cap, B, W), kept[idx])
        c = np.sort(ref[idx][:m])[::-1]
        if c[B - W - 1] - c[B - W] >= 1e-6:
            assert np.array_equal(oracle.select_topb(ref[idx], cap, B, W), kept[idx])
            checked += 1
        assert np.array_equal(Kg[idx][:B].view(np.uint16), host(K)[idx][kept[idx]].view(np.uint16))
    say("  %d of %d heads compared with the fp64 selection" % (checked, S * L * Hkv))
    assert checked >= S * L * Hkv // 2


def test_redundancy_full_shape_sampled():
    """7B heads at B = 512 (cap 641, 16 sequences): sampled heads against the oracle."""
    k = kvr()
    S, L, Hkv, D, B, W, buffer = 16, 28, 4, 128, 512, 128, 128
    cap = B + buffer + 1
    g = torch.Generator(device=DEV).manual_seed(5)
    K = torch.randn((S, L, Hkv, cap, D), generator=g, device=DEV).to(torch.bfloat16)
    imp = torch.rand((S, L, Hkv, cap), generator=g, device=DEV)
    out = torch.empty_like(imp)
    ln = torch.full((S,), cap, dtype=torch.int32, device=DEV)
    k.redundancy_scores(k.Cache(K, K, None), ln, imp, k.Policy(B, W, buffer), out)
    torch.cuda.synchronize()
    for (s, l, h) in ((0, 0, 0), (7, 13, 2), (15, 27, 3)):
        ref = rkv.rkv_head(host(K[s, l, h]), imp[s, l, h].double().cpu().numpy(), cap, W, 0.1, 7)
        got = out[s, l, h, : cap - W].double().cpu().numpy()
        np.testing.assert_allclose(got, ref, rtol=1e-4, atol=1e-6)
