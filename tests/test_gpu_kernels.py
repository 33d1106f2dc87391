"""GPU parity of each C-ABI entry point against the CPU oracle.

Inputs are seeded and drawn on the host, uploaded, consumed by the HIP kernels
through the C ABI (via the ctypes binding), and the very same host arrays go
to the oracle. Tolerances: attention outputs normwise per row within 2e-2
(bf16 storage, fp32 accumulation) or 1e-5 (fp32); importance scores within
1e-4 absolute; entropy within 1e-4 absolute; kept sets bit-exact on scores
separated by >= 1e-3 (and, for any scores, equal to the oracle's selection
applied to the GPU's own float32 scores).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from gpu_util import as_f64, host, rowwise_rel_err, say

pytestmark = pytest.mark.gpu

DEV = "cuda"
TOL = {torch.bfloat16: 2e-2, torch.float32: 1e-5}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_15797_amd import kvr  # noqa: F401  (fails loudly if libkvr.so is missing)
    yield


def kvr():
    from paper_2608_15797_amd import kvr as k
    return k


def randn(shape, g, dtype, std=1.0):
    return (torch.randn(shape, generator=g, dtype=torch.float32) * std).to(dtype)


# ------------------------------------------------------------ base attention

BASE_CASES = [
    # S, L, Hkv, G, D, B, W, buffer, dtype
    (3, 2, 1, 4, 64, 16, 8, 16, torch.float32),
    (3, 2, 2, 6, 128, 16, 4, 8, torch.float32),
    (4, 2, 4, 7, 128, 128, 32, 128, torch.bfloat16),
    (5, 3, 2, 8, 128, 64, 32, 64, torch.bfloat16),
    (3, 2, 2, 6, 64, 40, 8, 30, torch.bfloat16),
    (2, 1, 1, 16, 128, 20, 5, 7, torch.bfloat16),
    (2, 2, 3, 1, 128, 20, 5, 7, torch.bfloat16),
    # Cache shorter than one 32-key chunk, D = 64, with n = 1.
    (5, 1, 2, 4, 64, 12, 4, 6, torch.bfloat16),
    # Largest scored cache at G = 16: the window logits fill 61.6 KB of LDS (limit 64 KB).
    (2, 1, 1, 16, 128, 704, 64, 255, torch.bfloat16),
    # Group sizes that fill the 16-row tile partially in other ways.
    (3, 2, 2, 2, 128, 40, 8, 30, torch.bfloat16),
    (3, 2, 2, 3, 128, 40, 8, 30, torch.bfloat16),
    (2, 2, 2, 5, 64, 40, 8, 30, torch.bfloat16),
    (2, 1, 2, 9, 128, 40, 8, 30, torch.bfloat16),
    (2, 1, 2, 12, 128, 64, 32, 64, torch.bfloat16),
    (2, 1, 1, 15, 128, 40, 8, 30, torch.bfloat16),
]


@pytest.mark.parametrize("case", BASE_CASES, ids=lambda c: "S%dL%dHkv%dG%dD%d_B%dW%dbuf%d_%s" % (
    *c[:8], str(c[8]).split(".")[-1]))
def test_decode_attn_base_with_scores(case):
    """kvr_decode_attn on an evicted cache: append, attention (Eq. (1)) and the
    streamed window score for sequences before, at and inside the window."""
    S, L, Hkv, G, D, B, W, buffer, dt = case
    k = kvr()
    say("case", case)
    Hq = Hkv * G
    cap = B + buffer + 1
    g = torch.Generator().manual_seed(hash(case) & 0xffff)
    wstart = B + buffer + 2 - W
    # lengths: one not in the window, one at the first window step, others inside
    # the window, one at the overflow length, and n = 1.
    lens = [max(1, wstart - 3), wstart, min(cap, wstart + 5), cap, 1][:S]
    while len(lens) < S:
        lens.append(int(torch.randint(1, cap + 1, (1,), generator=g)))
    K = randn((S, L, Hkv, cap, D), g, dt)
    V = randn((S, L, Hkv, cap, D), g, dt)
    for s, n in enumerate(lens):  # stale slots must never be read
        K[s, :, :, n - 1:] = float("nan")
        V[s, :, :, n - 1:] = float("nan")
    q = randn((S, L, Hq, D), g, dt)
    kn = randn((S, L, Hkv, D), g, dt)
    vn = randn((S, L, Hkv, D), g, dt)
    new_pos = torch.arange(S, dtype=torch.int32) + 1000
    pos = torch.randint(0, 999, (S, L, Hkv, cap), generator=g, dtype=torch.int32)
    sc0 = torch.rand((S, L, Hkv, cap), generator=g) * 3
    scale = 1.0 / math.sqrt(D)

    cache = k.Cache(K.to(DEV), V.to(DEV), pos.to(DEV))
    lent = torch.tensor(lens, dtype=torch.int32, device=DEV)
    out = torch.empty((S, L, Hq, D), dtype=dt, device=DEV)
    scores = sc0.clone().to(DEV)
    k.decode_attn(cache, lent, q.to(DEV), out, scale, k_new=kn.to(DEV), v_new=vn.to(DEV),
                  new_pos=new_pos.to(DEV), policy=k.Policy(B, W, buffer), scores=scores)
    torch.cuda.synchronize()

    # Oracle: same cache with the new token appended on the host.
    Kh, Vh = K.clone(), V.clone()
    for s, n in enumerate(lens):
        Kh[s, :, :, n - 1] = kn[s]
        Vh[s, :, :, n - 1] = vn[s]
    ref, psum = oracle.decode_attn(host(Kh), host(Vh), np.array(lens), host(q), scale)

    # Append landed bit-exactly; pos written.
    Kg, Vg, posg = cache.k.cpu(), cache.v.cpu(), cache.pos.cpu()
    for s, n in enumerate(lens):
        assert torch.equal(Kg[s, :, :, n - 1].view(torch.int16) if dt == torch.bfloat16 else Kg[s, :, :, n - 1],
                           kn[s].view(torch.int16) if dt == torch.bfloat16 else kn[s])
        assert torch.equal(Vg[s, :, :, n - 1].float(), vn[s].float())
        assert (posg[s, :, :, n - 1] == 1000 + s).all()
        assert torch.equal(posg[s, :, :, : n - 1], pos[s, :, :, : n - 1])

    err = rowwise_rel_err(as_f64(out), ref)
    say("max rel err", err.max())
    assert err.max() <= TOL[dt], err.max()

    scg = scores.cpu().double().numpy()
    sc0n = sc0.double().numpy()
    for s, n in enumerate(lens):
        if n < wstart:
            assert np.array_equal(scg[s], sc0n[s]), "non-window sequence scores touched"
            continue
        if n == wstart:
            expect = psum[s, :, :, :n]
        else:
            expect = sc0.double().numpy()[s, :, :, :n] + psum[s, :, :, :n]
            expect[..., n - 1] = psum[s, :, :, n - 1]
        d = np.abs(scg[s, :, :, :n] - expect).max()
        say("seq", s, "n", n, "score err", d)
        assert d <= 1e-4
        # Converted: fp32 rounding of the stored prior adds at most 1 ulp of 3.
        assert np.array_equal(scg[s, :, :, n:], sc0n[s, :, :, n:])


def test_decode_attn_n1_returns_new_value():
    """n = 1: the output is the appended value (P6 special case on the GPU)."""
    k = kvr()
    S, L, Hkv, G, D, cap = 2, 1, 2, 7, 128, 17
    g = torch.Generator().manual_seed(5)
    cache = k.Cache.empty(S, L, Hkv, cap, D, torch.bfloat16, DEV)
    q = randn((S, L, Hkv * G, D), g, torch.bfloat16).to(DEV)
    kn = randn((S, L, Hkv, D), g, torch.bfloat16).to(DEV)
    vn = randn((S, L, Hkv, D), g, torch.bfloat16).to(DEV)
    out = torch.empty((S, L, Hkv * G, D), dtype=torch.bfloat16, device=DEV)
    k.decode_attn(cache, torch.ones(S, dtype=torch.int32, device=DEV), q, out, 0.1, k_new=kn,
                  v_new=vn)
    torch.cuda.synchronize()
    ref = vn.repeat_interleave(G, dim=2)
    assert torch.equal(out.cpu(), ref.cpu())


# ------------------------------------------------------------ helper (prefix)

PREFIX_CASES = [
    # S, P, L, Hkv, G, D, plen, scap, dtype
    (4, 4, 2, 2, 6, 128, 1000, 64, torch.bfloat16),   # private contexts, ragged plen
    (16, 2, 2, 2, 6, 128, 777, 40, torch.bfloat16),   # 8 candidates x 6 heads = 48 rows
    (8, 2, 1, 2, 8, 128, 2100, 33, torch.bfloat16),   # 4 x 8 = 32 rows
    (8, 1, 1, 1, 8, 128, 300, 16, torch.bfloat16),    # 8 x 8 = 64 rows
    (6, 3, 2, 2, 6, 64, 513, 20, torch.bfloat16),
    (8, 2, 2, 2, 6, 128, 150, 24, torch.bfloat16),    # spans of 512 keys cross up to 4 units
    (4, 2, 1, 2, 6, 128, 200, 24, torch.float32),
    # Row counts that are not multiples of 16: 3 x 5 = 15, 5 x 7 = 35, 13 x 3 = 39.
    (6, 2, 2, 2, 5, 128, 900, 20, torch.bfloat16),
    (10, 2, 1, 2, 7, 128, 700, 20, torch.bfloat16),
    (13, 1, 1, 2, 3, 64, 1100, 20, torch.bfloat16),
]


@pytest.mark.parametrize("case", PREFIX_CASES, ids=lambda c: "S%dP%dL%dHkv%dG%dD%d_plen%d_scap%d_%s" % (
    *c[:8], str(c[8]).split(".")[-1]))
def test_decode_attn_prefix(case):
    """Helper path: shared/private prefix then the candidate's own suffix, with
    ragged suffix lengths (split-K partials merged by log-sum-exp)."""
    S, P, L, Hkv, G, D, plen, scap, dt = case
    k = kvr()
    say("case", case)
    Hq = Hkv * G
    g = torch.Generator().manual_seed(plen * 7 + S)
    PK = randn((P, L, Hkv, plen, D), g, dt)
    PV = randn((P, L, Hkv, plen, D), g, dt)
    K = randn((S, L, Hkv, scap, D), g, dt)
    V = randn((S, L, Hkv, scap, D), g, dt)
    lens = torch.randint(1, scap + 1, (S,), generator=g, dtype=torch.int32)
    lens[0] = 1
    lens[-1] = scap
    q = randn((S, L, Hq, D), g, dt)
    kn = randn((S, L, Hkv, D), g, dt)
    vn = randn((S, L, Hkv, D), g, dt)
    scale = 1.0 / math.sqrt(D)
    cache = k.Cache(K.to(DEV), V.to(DEV), None)
    prefix = k.Prefix(PK.to(DEV), PV.to(DEV))
    nws = k.decode_attn_workspace_size(cache, prefix, Hq)
    ws = torch.full((max(nws, 16) // 4,), float("nan"), dtype=torch.float32, device=DEV)
    out = torch.empty((S, L, Hq, D), dtype=dt, device=DEV)
    k.decode_attn(cache, lens.to(DEV), q.to(DEV), out, scale, k_new=kn.to(DEV), v_new=vn.to(DEV),
                  prefix=prefix, workspace=ws)
    torch.cuda.synchronize()
    Kh, Vh = K.clone(), V.clone()
    for s in range(S):
        n = int(lens[s])
        Kh[s, :, :, n - 1] = kn[s]
        Vh[s, :, :, n - 1] = vn[s]
    ref, _ = oracle.decode_attn(host(Kh), host(Vh), lens.numpy(), host(q), scale,
                                prefix_K=host(PK), prefix_V=host(PV), want_psum=False)
    err = rowwise_rel_err(as_f64(out), ref)
    say("max rel err", err.max(), "workspace bytes", nws)
    assert err.max() <= TOL[dt]


def test_prefix_workspace_errors():
    k = kvr()
    cache = k.Cache.empty(4, 1, 2, 8, 128, torch.bfloat16, DEV, with_pos=False)
    prefix = k.Prefix(torch.zeros((2, 1, 2, 64, 128), dtype=torch.bfloat16, device=DEV),
                      torch.zeros((2, 1, 2, 64, 128), dtype=torch.bfloat16, device=DEV))
    out = torch.empty((4, 1, 12, 128), dtype=torch.bfloat16, device=DEV)
    q = torch.zeros_like(out)
    with pytest.raises(k.KvrError) as e:
        k.decode_attn(cache, torch.ones(4, dtype=torch.int32, device=DEV), q, out, 1.0,
                      prefix=prefix)
    assert e.value.status == -4


# ------------------------------------------------------------ eviction

def planted_scores(shape, n, g):
    """Per head a random permutation of c + 2e-3*k + U(0, 5e-4): pairwise gaps
    >= 1.5e-3, so the kept set is unique and must match bit for bit."""
    S, L, Hkv, cap = shape
    sc = torch.zeros(shape, dtype=torch.float32)
    base = torch.arange(n, dtype=torch.float64) * 2e-3
    for s in range(S):
        for l in range(L):
            for h in range(Hkv):
                perm = torch.randperm(n, generator=g)
                sc[s, l, h, :n] = (0.5 + base[perm] + torch.rand(n, generator=g, dtype=torch.float64) * 5e-4).float()
    return sc


EVICT_CASES = [
    # S, L, Hkv, D, B, W, buffer, dtype
    (3, 2, 2, 64, 16, 8, 16, torch.float32),
    (4, 3, 4, 128, 128, 32, 128, torch.bfloat16),
    (6, 2, 8, 128, 64, 32, 64, torch.bfloat16),
    (3, 2, 2, 128, 20, 5, 7, torch.float32),
    # An 8000-slot cache (the commit path's one-shot compression): candidates past
    # the select's registers, read back from LDS.
    (1, 1, 2, 128, 256, 32, 7743, torch.bfloat16),
    # Largest cache the eviction kernel takes at B = 256: cap + B = 16384 slots,
    # 64 KiB of LDS for the keys and the kept set.
    (1, 1, 2, 128, 256, 32, 15871, torch.bfloat16),
]


@pytest.mark.parametrize("case", EVICT_CASES, ids=lambda c: "S%dL%dHkv%dD%d_B%dW%dbuf%d_%s" % (
    *c[:7], str(c[7]).split(".")[-1]))
def test_evict_topb_planted(case):
    """kvr_evict_topb: kept sets bit-exact against the oracle's TopB on
    separated scores; K, V, pos compacted bit-exactly; sequences below the
    bound untouched."""
    S, L, Hkv, D, B, W, buffer, dt = case
    k = kvr()
    say("case", case)
    cap = B + buffer + 1
    g = torch.Generator().manual_seed(B * 31 + S)
    lens = [cap if s % 2 == 0 else cap - 1 - s for s in range(S)]
    K = randn((S, L, Hkv, cap, D), g, dt)
    V = randn((S, L, Hkv, cap, D), g, dt)
    pos = torch.arange(cap, dtype=torch.int32).repeat(S, L, Hkv, 1) + 7
    sc = planted_scores((S, L, Hkv, cap), cap - W, g)
    cache = k.Cache(K.clone().to(DEV), V.clone().to(DEV), pos.clone().to(DEV))
    kept = torch.full((S, L, Hkv, B), -1, dtype=torch.int32, device=DEV)
    len_out = torch.full((S,), -7, dtype=torch.int32, device=DEV)
    k.evict_topb(cache, torch.tensor(lens, dtype=torch.int32, device=DEV), sc.to(DEV),
                 k.Policy(B, W, buffer), kept=kept, len_out=len_out)
    torch.cuda.synchronize()
    assert len_out.cpu().tolist() == [B if n > B + buffer else n for n in lens]
    Kg, Vg, pg, kg = host(cache.k), host(cache.v), cache.pos.cpu().numpy(), kept.cpu().numpy()
    Kh, Vh, ph = host(K).copy(), host(V).copy(), pos.numpy().copy()
    scn = sc.double().numpy()
    for s in range(S):
        n = lens[s]
        for l in range(L):
            for h in range(Hkv):
                if n <= B + buffer:
                    assert (kg[s, l, h] == -1).all()
                    continue
                ref = oracle.select_topb(scn[s, l, h], n, B, W)
                assert np.array_equal(kg[s, l, h], ref), (s, l, h)
                oracle.compact_head(Kh[s, l, h], Vh[s, l, h], ph[s, l, h], ref)
    assert np.array_equal(Kg.view(np.uint8), Kh.view(np.uint8))
    assert np.array_equal(Vg.view(np.uint8), Vh.view(np.uint8))
    assert np.array_equal(pg, ph)


@pytest.mark.parametrize("S,L,Hkv,B,W,buffer", [(64, 28, 4, 128, 32, 128), (32, 80, 8, 64, 32, 64)])
def test_evict_topb_planted_full_shape(S, L, Hkv, B, W, buffer):
    """Full workload shapes (7B: 64 x 28 x 4 heads, cap 257; 72B: 32 x 80 x 8,
    cap 129) with planted scores separated by >= 1.5e-3: every kept set equals
    the oracle's bit for bit, and the compaction moves exactly those rows."""
    k = kvr()
    D, cap = 128, B + buffer + 1
    g = torch.Generator().manual_seed(S * L + B)
    n = cap - W
    base = torch.arange(n, dtype=torch.float64) * 2e-3
    perm = torch.argsort(torch.rand((S, L, Hkv, n), generator=g), dim=-1)
    sc = torch.zeros((S, L, Hkv, cap), dtype=torch.float32)
    sc[..., :n] = (0.5 + base[perm] + torch.rand((S, L, Hkv, n), generator=g, dtype=torch.float64) * 5e-4).float()
    # Row j of every head holds the value j in all of its elements, so the
    # compacted cache reveals which rows moved where.
    rowid = torch.arange(cap, dtype=torch.float32).view(1, 1, 1, cap, 1)
    K = (rowid * 0.5).expand(S, L, Hkv, cap, D).to(torch.bfloat16).contiguous()
    V = (rowid * 0.25).expand(S, L, Hkv, cap, D).to(torch.bfloat16).contiguous()
    cache = k.Cache(K.to(DEV), V.to(DEV), torch.arange(cap, dtype=torch.int32).repeat(S, L, Hkv, 1).to(DEV))
    kept = torch.empty((S, L, Hkv, B), dtype=torch.int32, device=DEV)
    k.evict_topb(cache, torch.full((S,), cap, dtype=torch.int32, device=DEV), sc.to(DEV),
                 k.Policy(B, W, buffer), kept=kept)
    torch.cuda.synchronize()
    kg = kept.cpu().numpy()
    scn = sc.double().numpy()
    for idx in np.ndindex(S, L, Hkv):
        ref = oracle.select_topb(scn[idx], cap, B, W)
        assert np.array_equal(kg[idx], ref), idx
    assert np.array_equal(cache.pos.cpu().numpy()[..., :B], kg)
    Kg = cache.k[..., :B, :].float().cpu()
    assert torch.equal(Kg, (torch.from_numpy(kg).float() * 0.5)[..., None].expand_as(Kg).to(torch.bfloat16).float())


@pytest.mark.parametrize("B,W,buffer,levels", [(24, 6, 10, 3), (128, 32, 300, 5), (64, 32, 64, 1)])
def test_evict_topb_ties_and_gpu_scores_selection(B, W, buffer, levels):
    """Exact ties go to the lower slot (integer-valued scores, signed and
    with -0 next to +0); 97 candidates (select keys in registers) and 397
    (keys re-read from LDS); one level: every score equal."""
    k = kvr()
    S, L, Hkv, D = 2, 2, 2, 128
    cap = B + buffer + 1
    g = torch.Generator().manual_seed(77 + buffer)
    sc = (torch.randint(0, levels, (S, L, Hkv, cap), generator=g) - levels // 2).float()
    sc[0, 0, 0, ::7] = -0.0
    cache = k.Cache.empty(S, L, Hkv, cap, D, torch.bfloat16, DEV)
    kept = torch.empty((S, L, Hkv, B), dtype=torch.int32, device=DEV)
    k.evict_topb(cache, torch.full((S,), cap, dtype=torch.int32, device=DEV), sc.to(DEV),
                 k.Policy(B, W, buffer), kept=kept)
    torch.cuda.synchronize()
    for s in range(S):
        for l in range(L):
            for h in range(Hkv):
                ref = oracle.select_topb(sc[s, l, h].double().numpy(), cap, B, W)
                assert np.array_equal(kept[s, l, h].cpu().numpy(), ref)


# ------------------------------------------------------------ window scores

@pytest.mark.parametrize("dt,D,G,nq,cap", [
    (torch.float32, 64, 4, 8, 97),
    (torch.bfloat16, 128, 7, 32, 97),
    (torch.bfloat16, 128, 8, 5, 97),
    (torch.bfloat16, 64, 4, 8, 97),
    (torch.bfloat16, 128, 16, 33, 130),    # 33 row blocks: the last pair is half empty
    (torch.bfloat16, 128, 1, 3, 40),       # fewer rows than one block
    (torch.bfloat16, 128, 7, 128, 300),    # a committed step's window on the 7B head shape
    (torch.bfloat16, 128, 4, 8, 6144),     # largest cache of the LDS-ring kernel: 64-bit accumulator + ring = 64 KB
    (torch.bfloat16, 64, 4, 8, 7500),      # beyond it at D = 64: the single-wave-stream kernel
    (torch.bfloat16, 128, 4, 8, 8192),     # largest cache: the accumulator alone fills 64 KB of LDS
])
def test_accumulate_scores(dt, D, G, nq, cap):
    """kvr_accumulate_scores equals the oracle's causal window re-computation,
    in both overwrite and accumulate modes; lengths include the full cache, a
    ragged one, nq + 1 and fewer than nq (early window rows then see nothing)."""
    k = kvr()
    S, L, Hkv = 4, 2, 2
    g = torch.Generator().manual_seed(D + G + nq)
    K = randn((S, L, Hkv, cap, D), g, dt)
    V = randn((S, L, Hkv, cap, D), g, dt)
    lens = [cap, min(50, cap - 3), min(nq + 1, cap), max(1, min(nq - 2, cap))]
    qw = randn((S, L, Hkv * G, nq, D), g, dt)
    scale = 1.0 / math.sqrt(D)
    cache = k.Cache(K.to(DEV), V.to(DEV), None)
    lent = torch.tensor(lens, dtype=torch.int32, device=DEV)
    sc = torch.full((S, L, Hkv, cap), 0.25, device=DEV)
    k.accumulate_scores(cache, lent, qw.to(DEV), scale, sc, accumulate=False)
    torch.cuda.synchronize()
    ref = oracle.window_scores(host(K), host(V), np.array(lens), host(qw), scale)
    got = sc.cpu().double().numpy()
    for s, n in enumerate(lens):
        assert np.abs(got[s, ..., :n] - ref[s, ..., :n]).max() <= 1e-4
        assert (got[s, ..., n:] == 0.25).all()
    first = sc.clone()
    k.accumulate_scores(cache, lent, qw.to(DEV), scale, sc, accumulate=True)
    torch.cuda.synchronize()
    got = sc.cpu().double().numpy()
    for s, n in enumerate(lens):
        assert np.abs(got[s, ..., :n] - 2 * ref[s, ..., :n]).max() <= 2e-4
    # Bitwise reproducible: the same call again gives the same bits (the
    # column sums of the workgroup's waves are added in fixed point).
    for _ in range(3):
        again = torch.full((S, L, Hkv, cap), 0.25, device=DEV)
        k.accumulate_scores(cache, lent, qw.to(DEV), scale, again, accumulate=False)
        torch.cuda.synchronize()
        assert torch.equal(again.view(torch.int32), first.view(torch.int32))


# ------------------------------------------------------------ entropy

ENT_CASES = [
    # R, V, ld, dtype, std
    (1, 1, 8, torch.float32, 1.0),
    (3, 7, 7, torch.float32, 2.0),
    (1, 1024, 1024, torch.float32, 2.0),
    (8, 151936, 151936, torch.bfloat16, 3.0),
    (64, 152064, 152064, torch.bfloat16, 3.0),
    (5, 152064, 152072, torch.bfloat16, 0.1),
    (300, 1000, 1003, torch.bfloat16, 1.0),
    (2, 50000, 50000, torch.float32, 5.0),
    (300, 152064, 152064, torch.bfloat16, 3.0),  # whole-row workgroups
]


@pytest.mark.parametrize("case", ENT_CASES, ids=lambda c: "R%dV%dld%d_%s" % (
    c[0], c[1], c[2], str(c[3]).split(".")[-1]))
def test_logit_entropy(case):
    k = kvr()
    R, V, ld, dt, std = case
    g = torch.Generator().manual_seed(R * 13 + V)
    x = torch.zeros((R, ld), dtype=torch.float32)
    x[:, :V] = torch.randn((R, V), generator=g) * std
    if V > 20:
        x[0, 3:9] = float("-inf")
        x[-1, :5] += 10.0
    x[:, V:] = 1e3  # padding must be ignored
    xd = x.to(dt)
    H = torch.empty(R, device=DEV)
    ws = torch.zeros(max(k.logit_entropy_workspace_size(R, V), 16) // 4, device=DEV)
    xg = xd.to(DEV)
    for rep in range(2):  # workspace counters must reset between calls
        H.fill_(float("nan"))
        k.logit_entropy(xg, H, V=V, workspace=ws)
        torch.cuda.synchronize()
        ref = oracle.entropy(host(xd), V=V)
        d = np.abs(H.cpu().double().numpy() - ref).max()
        say("rep", rep, "max abs err", d)
        assert d <= 1e-4
    # inv_temp
    k.logit_entropy(xg, H, V=V, inv_temp=1.25, workspace=ws)
    torch.cuda.synchronize()
    ref = oracle.entropy(host(xd), V=V, inv_temp=1.25)
    assert np.abs(H.cpu().double().numpy() - ref).max() <= 1e-4


ENT_BATCH_CASES = [
    # per set: R, V, ld, std, inv_temp, with detector
    [(128, 152064, 152064, 3.0, 1.0, True), (128, 151936, 151936, 1.0, 1.25, False)],
    [(1, 1000, 1000, 1.0, 1.0, False), (64, 152064, 152064, 0.1, 1.0, True),
     (5, 2048, 2048, 2.0, 0.8, True), (300, 8000, 8000, 3.0, 1.0, False)],
    [(3, 7, 9, 2.0, 1.0, False), (1, 1, 1, 1.0, 1.0, False), (4, 50000, 50003, 5.0, 1.0, True)],
    [(32, 152064, 152064, 3.0, 1.0, True)],
    # At least 256 long rows: one whole-row workgroup per row; the second set's
    # stride is not a multiple of 16 bytes, so every set takes the scalar loads.
    [(200, 152064, 152064, 3.0, 1.0, True), (57, 100000, 100003, 1.0, 1.25, True)],
]


@pytest.mark.parametrize("ci", range(len(ENT_BATCH_CASES)))
@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
def test_logit_entropy_batch(ci, dt):
    """One launch over several sets of rows (different vocabularies, strides,
    temperatures and detectors): every set's entropies match the oracle, and
    each detector holds exactly its own set's history."""
    k = kvr()
    specs = ENT_BATCH_CASES[ci]
    g = torch.Generator().manual_seed(71 + ci)
    sets, hosts, odets = [], [], []
    for j, (R, V, ld, std, it, with_det) in enumerate(specs):
        x = torch.full((R, ld), 1e3)  # padding must be ignored
        x[:, :V] = torch.randn((R, V), generator=g) * std
        if V > 20:
            x[0, 3:9] = float("-inf")
            x[-1, :5] += 10.0
        xd = x.to(dt)
        det = k.Detector.zeros(R, window=12, guard=3, tau=5.0, device=DEV) if with_det else None
        sets.append(k.LogitSet(xd.to(DEV), torch.full((R,), float("nan"), device=DEV), V, it, det))
        hosts.append(xd)
        odets.append(oracle.Detector(R, window=12, guard=3, tau=5.0) if with_det else None)
    need = k.logit_entropy_batch_workspace_size([(s[0], s[1]) for s in specs], dt)
    ws = torch.zeros(max(need, 16) // 4, device=DEV)
    say("case", ci, "sets", [(s[0], s[1]) for s in specs], "workspace", need)
    for rep in range(4):  # the workspace needs no reset between calls
        for s in sets:
            s.H.fill_(float("nan"))
        k.logit_entropy_batch(sets, workspace=ws)
        torch.cuda.synchronize()
        for j, (s, xh, od) in enumerate(zip(sets, hosts, odets)):
            ref = oracle.entropy(host(xh), V=specs[j][1], inv_temp=specs[j][4])
            got = s.H.cpu().double().numpy()
            d = np.abs(got - ref).max()
            say("rep", rep, "set", j, "max abs err", d)
            assert d <= 1e-4
            if od is not None:
                fref = od.step(ref)
                assert s.detector.cnt.cpu().numpy().tolist() == [rep + 1] * specs[j][0]
                f = s.detector.flag.cpu().numpy()
                for r in range(specs[j][0]):
                    mean = od.hist[r, :min(int(od.cnt[r]), 12)].mean()
                    if od.cnt[r] >= 3 and abs(mean - 5.0) < 1e-4:
                        continue
                    assert f[r] == fref[r], (rep, j, r)


def test_entropy_closed_forms_on_gpu():
    k = kvr()
    V = 152064
    x = torch.zeros((3, V), dtype=torch.bfloat16)
    x[1] = float("-inf")
    x[1, 12345] = 3.0
    x[2, :5] = 10.0
    H = torch.empty(3, device=DEV)
    ws = torch.zeros(max(k.logit_entropy_workspace_size(3, V), 16) // 4, device=DEV)
    k.logit_entropy(x.to(DEV), H, workspace=ws)
    torch.cuda.synchronize()
    h = H.cpu().double().numpy()
    assert abs(h[0] - math.log(V)) <= 1e-4
    assert abs(h[1]) <= 1e-6
    d = 10.0
    Z = 5 * math.exp(d) + (V - 5)
    assert abs(h[2] - (math.log(Z) - 5 * d * math.exp(d) / Z)) <= 1e-4


def test_entropy_detector_on_gpu():
    """Detector epilogue: high-entropy rows fire at the guard position, low
    rows never; the oracle detector fed the oracle entropies agrees wherever
    the moving mean is not within 1e-4 of tau."""
    k = kvr()
    R, V = 6, 2048
    g = torch.Generator().manual_seed(9)
    det = k.Detector.zeros(R, window=12, guard=24, tau=7.0, device=DEV)
    odet = oracle.Detector(R, window=12, guard=24, tau=7.0)
    H = torch.empty(R, device=DEV)
    for pos in range(40):
        x = torch.randn((R, V), generator=g) * torch.tensor([0.1, 0.5, 1.0, 2.0, 3.0, 0.05])[:, None]
        if pos > 30:
            x[5] *= 100
        xd = x.to(torch.bfloat16)
        k.logit_entropy(xd.to(DEV), H, detector=det)
        torch.cuda.synchronize()
        href = oracle.entropy(host(xd))
        fref = odet.step(href)
        mean = odet.hist.mean(axis=1)
        f = det.flag.cpu().numpy()
        for r in range(R):
            if odet.cnt[r] >= 24 and abs(mean[r] - 7.0) < 1e-4:
                continue
            assert f[r] == fref[r], (pos, r, mean[r])
    assert det.cnt.cpu().numpy().tolist() == [40] * R
