"""kvr_decode_attn_entropy: base attention and the step's entropies in one
launch, through the C ABI.

The same inputs go through the fused call and through the two separate calls
(kvr_decode_attn, then kvr_logit_entropy_batch): attention outputs, streamed
scores and the appended cache rows must be bit for bit those of
kvr_decode_attn (the attention lanes of the fused launch run the same code);
every entropy must be within 1e-4 of the oracle, and the detector state
(history, counts, flags) must follow the oracle's detector over three calls.
Cases cover both cache types, bf16 and float32 logits, several sets with
their own vocabulary, stride and temperature, a vocabulary below one 8-logit
vector and one that is not a multiple of 8, -inf entries and a boosted row.

With a prefix (the helper path) the rows ride in the context launch, whose
split plan leaves their waves slots of their own: the outputs there are
compared with the oracle at the helper path's tolerance, the appended rows
bit for bit with kvr_decode_attn's.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from gpu_util import as_f64, host, rowwise_rel_err, say

pytestmark = pytest.mark.gpu

DEV = "cuda"

CASES = [
    # cache (S, L, Hkv, G, D, B, W, buffer, dtype), logit dtype, sets [(R, V, ld, std, inv_temp, detector)]
    ((4, 2, 4, 7, 128, 64, 32, 64, torch.bfloat16), torch.bfloat16,
     [(16, 152064, 152064, 3.0, 1.0, True), (9, 151936, 152000, 1.0, 0.7, False)]),
    ((3, 2, 2, 8, 128, 16, 4, 8, torch.bfloat16), torch.float32,
     [(5, 1023, 1024, 2.0, 1.0, True), (3, 5, 8, 1.0, 1.0, False), (2, 8, 8, 0.5, 2.0, True)]),
    ((2, 1, 2, 4, 64, 12, 4, 6, torch.bfloat16), torch.bfloat16, [(7, 50000, 50000, 2.0, 1.0, True)]),
    ((1, 1, 1, 4, 64, 16, 8, 16, torch.float32), torch.float32, [(1, 1024, 1024, 2.0, 1.0, True)]),
]


def _randn(shape, g, dtype, std=1.0):
    return (torch.randn(shape, generator=g, dtype=torch.float32) * std).to(dtype)


@pytest.mark.parametrize("ci", range(len(CASES)))
def test_decode_attn_entropy_matches_separate_calls(ci):
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_15797_amd import kvr as k
    (S, L, Hkv, G, D, B, W, buffer, dt), ldt, specs = CASES[ci]
    say("case", ci, "cache", CASES[ci][0], "logits", ldt, "sets", specs)
    Hq = Hkv * G
    cap = B + buffer + 1
    wstart = B + buffer + 2 - W
    g = torch.Generator().manual_seed(4242 + ci)
    scale = 1.0 / math.sqrt(D)
    K = _randn((S, L, Hkv, cap, D), g, dt)
    V = _randn((S, L, Hkv, cap, D), g, dt)
    pos = torch.randint(0, 999, (S, L, Hkv, cap), generator=g, dtype=torch.int32)
    sc0 = torch.rand((S, L, Hkv, cap), generator=g) * 3
    pol = k.Policy(B, W, buffer)

    def caches():
        return [k.Cache(K.to(DEV), V.to(DEV), pos.to(DEV)) for _ in range(2)]

    ca, cb = caches()
    sa, sb = sc0.to(DEV), sc0.to(DEV)
    # Logit rows (with padding past V that must be ignored) and detectors.
    xs = []
    for R, V_, ld, std, it, det in specs:
        x = torch.full((R, ld), 1e3)
        x[:, :V_] = torch.randn((R, V_), generator=g) * std
        if V_ > 20:
            x[0, 3:9] = float("-inf")
            x[-1, :5] += 10.0
        xs.append(x.to(ldt))

    def sets(tag):
        return [k.LogitSet(x.to(DEV), torch.full((x.shape[0],), float("nan"), device=DEV), V_, it,
                           k.Detector.zeros(x.shape[0], window=12, guard=1, tau=5.0, device=DEV) if det else None)
                for x, (R, V_, ld, std, it, det) in zip(xs, specs)]

    seta, setb = sets("a"), sets("b")
    odets = [oracle.Detector(R, window=12, guard=1, tau=5.0) if det else None for R, V_, ld, std, it, det in specs]
    need = k.logit_entropy_batch_workspace_size([(R, V_) for R, V_, *_ in specs], ldt)
    ws = torch.zeros(max(need, 16) // 4, device=DEV)
    Href = [oracle.entropy(host(x), V=V_, inv_temp=it) for x, (R, V_, ld, std, it, det) in zip(xs, specs)]
    for step in range(3):
        # Lengths: before, at and inside the observation window.
        lens = [max(1, wstart - 2 + step), wstart + step, min(cap, wstart + 3 + step)][:S]
        while len(lens) < S:
            lens.append(min(cap, 1 + 7 * len(lens) + step))
        lent = torch.tensor(lens, dtype=torch.int32, device=DEV)
        q = _randn((S, L, Hq, D), g, dt).to(DEV)
        kn = _randn((S, L, Hkv, D), g, dt).to(DEV)
        vn = _randn((S, L, Hkv, D), g, dt).to(DEV)
        npos = (torch.arange(S, dtype=torch.int32) + 1000 + step).to(DEV)
        oa = torch.empty((S, L, Hq, D), dtype=dt, device=DEV)
        ob = torch.empty_like(oa)
        k.decode_attn(ca, lent, q, oa, scale, k_new=kn, v_new=vn, new_pos=npos, policy=pol, scores=sa)
        k.logit_entropy_batch(seta, workspace=ws)
        k.decode_attn_entropy(cb, lent, q, ob, scale, setb, k_new=kn, v_new=vn, new_pos=npos, policy=pol,
                              scores=sb)
        torch.cuda.synchronize()
        assert torch.equal(oa.cpu().view(torch.int16) if dt == torch.bfloat16 else oa.cpu(),
                           ob.cpu().view(torch.int16) if dt == torch.bfloat16 else ob.cpu())
        assert torch.equal(sa.cpu(), sb.cpu())
        for t in ("k", "v"):
            x, y = getattr(ca, t).cpu(), getattr(cb, t).cpu()
            assert torch.equal(x.view(torch.int16) if dt == torch.bfloat16 else x,
                               y.view(torch.int16) if dt == torch.bfloat16 else y)
        assert torch.equal(ca.pos.cpu(), cb.pos.cpu())
        for j, (a, b, ref, od) in enumerate(zip(seta, setb, Href, odets)):
            hb = b.H.cpu().double().numpy()
            d = np.abs(hb - ref).max()
            say("  step", step, "set", j, "max |fused - oracle|", d, "max |fused - batch|",
                np.abs(hb - a.H.cpu().double().numpy()).max())
            assert d <= 1e-4
            if od is not None:
                fref = od.step(ref)
                assert b.detector.cnt.cpu().numpy().tolist() == [step + 1] * len(ref)
                assert np.abs(b.detector.hist.cpu().double().numpy()[:, step] - ref).max() <= 1e-4
                # Flags may differ only where the moving mean lies within 1e-4 of tau.
                mean = od.hist[:, : step + 1].mean(axis=1)
                f = b.detector.flag.cpu().numpy()
                ok = (f == fref) | (np.abs(mean - 5.0) < 1e-4)
                assert ok.all()


def test_decode_attn_entropy_rejects_unaligned_rows():
    from paper_2608_15797_amd import kvr as k
    S, L, Hkv, G, D, cap = 2, 1, 1, 4, 128, 33
    cache = k.Cache.empty(S, L, Hkv, cap, D, torch.bfloat16, DEV)
    q = torch.zeros((S, L, Hkv * G, D), dtype=torch.bfloat16, device=DEV)
    out = torch.empty_like(q)
    lent = torch.ones(S, dtype=torch.int32, device=DEV)
    x = torch.zeros((4, 1001), dtype=torch.bfloat16, device=DEV)  # ld * 2 = 2002 bytes
    with pytest.raises(k.KvrError) as e:
        k.decode_attn_entropy(cache, lent, q, out, 1.0, [k.LogitSet(x, torch.empty(4, device=DEV))])
    assert e.value.status == -1 and "aligned" in str(e.value)


SAMPLE_CASES = [
    # cache (S, L, Hkv, G, D, B, W, buffer, dtype), logit dtype, sets [(R, V, ld, kind)], sampler (T, k, p, seed, step)
    ((4, 2, 4, 7, 128, 64, 32, 64, torch.bfloat16), torch.bfloat16,
     [(16, 152064, 152064, "boosted"), (9, 151936, 152000, "ties")], (0.8, 20, 0.95, 1234, 7)),
    ((3, 2, 2, 8, 128, 16, 4, 8, torch.bfloat16), torch.float32,
     [(5, 1023, 1024, 2.0), (3, 5, 8, 1.0), (2, 8, 8, "flat")], (1.0, 64, 1.0, 9, 0)),
    ((1, 1, 1, 4, 64, 16, 8, 16, torch.float32), torch.bfloat16, [(4, 1024, 1024, 2.0)], (0.5, 1, 0.5, 3, 2)),
]


@pytest.mark.parametrize("ci", range(len(SAMPLE_CASES)))
def test_decode_attn_entropy_sample_matches_separate_calls(ci):
    """kvr_decode_attn_entropy_sample: attention bit for bit as
    kvr_decode_attn, entropies within 1e-4 of the oracle, and every set's
    tokens identical to kvr_logit_entropy_sample's on the same rows and
    settings (same k best logits, same draw), which in turn follow the
    oracle sampler (oracle/sampler.py) as in test_gpu_sampler."""
    from paper_2608_15797_amd import kvr as k
    from test_gpu_sampler import _check_tokens, _logits
    (S, L, Hkv, G, D, B, W, buffer, dt), ldt, specs, (T, topk, topp, seed, step) = SAMPLE_CASES[ci]
    say("case", ci, "cache", SAMPLE_CASES[ci][0], "logits", ldt, "sets", specs)
    Hq = Hkv * G
    cap = B + buffer + 1
    g = torch.Generator().manual_seed(5151 + ci)
    scale = 1.0 / math.sqrt(D)
    K = _randn((S, L, Hkv, cap, D), g, dt)
    V = _randn((S, L, Hkv, cap, D), g, dt)
    pos = torch.randint(0, 999, (S, L, Hkv, cap), generator=g, dtype=torch.int32)
    pol = k.Policy(B, W, buffer)
    smp = k.Sampler(temperature=T, top_k=topk, top_p=topp, seed=seed, step=step)
    xs = [_logits(R, V_, ld, ldt, kind, 77 + j) for j, (R, V_, ld, kind) in enumerate(specs)]
    lens = [min(cap, B + buffer + 2 - W + s) for s in range(S)]
    lent = torch.tensor(lens, dtype=torch.int32, device=DEV)
    q = _randn((S, L, Hq, D), g, dt).to(DEV)
    kn = _randn((S, L, Hkv, D), g, dt).to(DEV)
    vn = _randn((S, L, Hkv, D), g, dt).to(DEV)
    npos = (torch.arange(S, dtype=torch.int32) + 2000).to(DEV)
    sc0 = torch.rand((S, L, Hkv, cap), generator=g)
    ca = k.Cache(K.to(DEV), V.to(DEV), pos.to(DEV))
    cb = k.Cache(K.to(DEV), V.to(DEV), pos.to(DEV))
    sa, sb = sc0.to(DEV), sc0.to(DEV)
    oa = torch.empty((S, L, Hq, D), dtype=dt, device=DEV)
    ob = torch.empty_like(oa)
    k.decode_attn(ca, lent, q, oa, scale, k_new=kn, v_new=vn, new_pos=npos, policy=pol, scores=sa)
    ref_tok = []
    for x, (R, V_, ld, kind) in zip(xs, specs):
        H = torch.empty(R, device=DEV)
        tok = torch.full((R,), -7, dtype=torch.int32, device=DEV)
        ws = torch.empty(max(k.logit_entropy_sample_workspace_size(R, V_, topk), 16) // 4 + 4, device=DEV)
        k.logit_entropy_sample(x.to(DEV), H, tok, smp, V=V_, workspace=ws)
        ref_tok.append(tok)
    sets = [k.LogitSet(x.to(DEV), torch.full((x.shape[0],), float("nan"), device=DEV), V_, 1.0)
            for x, (R, V_, ld, kind) in zip(xs, specs)]
    toks = [torch.full((x.shape[0],), -7, dtype=torch.int32, device=DEV) for x in xs]
    k.decode_attn_entropy_sample(cb, lent, q, ob, scale, sets, smp, toks, k_new=kn, v_new=vn, new_pos=npos,
                                 policy=pol, scores=sb)
    torch.cuda.synchronize()
    bits = (lambda t: t.cpu().view(torch.int16)) if dt == torch.bfloat16 else (lambda t: t.cpu())
    assert torch.equal(bits(oa), bits(ob))
    assert torch.equal(sa.cpu(), sb.cpu())
    for t in ("k", "v"):
        assert torch.equal(bits(getattr(ca, t)), bits(getattr(cb, t)))
    for j, (x, (R, V_, ld, kind)) in enumerate(zip(xs, specs)):
        got = toks[j].cpu().numpy()
        assert (got == ref_tok[j].cpu().numpy()).all(), (j, got, ref_tok[j].cpu().numpy())
        exact, loose = _check_tokens(host(x), V_, smp, got)
        href = oracle.entropy(host(x), V=V_)
        d = np.abs(sets[j].H.cpu().double().numpy() - href).max()
        say("  set", j, "tokens", got[:8].tolist(), "oracle-exact", exact, "near-threshold", loose, "H err", d)
        assert d <= 1e-4


PREFIX_CASES = [
    # helper (S, P, L, Hkv, G, D, plen, scap, dtype), logit dtype, sets [(R, V, ld, kind, detector)], sampler
    # Private 4096-token contexts of the helper-only workload's shape, 8 rows of its vocabulary.
    ((8, 8, 2, 2, 6, 128, 4096, 40, torch.bfloat16), torch.bfloat16, [(8, 151936, 151936, "boosted", True)], None),
    # 8 candidates x 6 heads share each context (three row blocks); float32 logits, two sets.
    ((16, 2, 2, 2, 6, 128, 777, 40, torch.bfloat16), torch.float32,
     [(5, 1023, 1024, "2.0", True), (3, 5, 8, "1.0", False)], None),
    # Head dim 64, spans crossing units; the sampler draws every row's token.
    ((6, 3, 2, 2, 6, 64, 513, 20, torch.bfloat16), torch.bfloat16,
     [(6, 4099, 4104, "boosted", False), (2, 151936, 151936, "ties", False)], (0.8, 20, 0.95, 77, 3)),
    # More rows than half the chip's context waves (1024 at one row block): the
    # plan keeps 512 for the 524288 context keys (spans of 1024 keys, not 512).
    ((4, 4, 4, 2, 6, 128, 16384, 16, torch.bfloat16), torch.bfloat16, [(1500, 64, 64, "2.0", False)], None),
    # 4 candidates x 8 heads (two row blocks) and 8 x 8 (four row blocks, the kernel that spills to scratch).
    ((8, 2, 1, 2, 8, 128, 2100, 33, torch.bfloat16), torch.bfloat16, [(3, 151936, 151936, "boosted", True)], None),
    ((8, 1, 1, 1, 8, 128, 300, 16, torch.bfloat16), torch.float32, [(4, 5000, 5000, "2.0", False)],
     (0.8, 20, 0.95, 5, 1)),
    # float32 caches: the entropy rows run as a kernel of their own after the attention kernel.
    ((4, 2, 2, 2, 6, 128, 200, 24, torch.float32), torch.float32, [(4, 1024, 1024, "2.0", True)], None),
]


@pytest.mark.parametrize("ci", range(len(PREFIX_CASES)))
def test_decode_attn_entropy_with_prefix(ci):
    """kvr_decode_attn_entropy(_sample) with a prefix: the logit rows ride in
    the context launch. Attention outputs within the helper path's tolerance
    of the oracle (the split points differ from kvr_decode_attn's, so the
    outputs agree with it to rounding, not bit for bit), the appended suffix
    rows bit for bit, entropies within 1e-4 of the oracle, the detector as
    the oracle's, and the tokens those of kvr_logit_entropy_sample."""
    from paper_2608_15797_amd import kvr as k
    from test_gpu_sampler import _check_tokens, _logits
    (S, P, L, Hkv, G, D, plen, scap, dt), ldt, specs, smp_args = PREFIX_CASES[ci]
    say("case", ci, "helper", PREFIX_CASES[ci][0], "logits", ldt, "sets", specs, "sampler", smp_args)
    Hq = Hkv * G
    g = torch.Generator().manual_seed(6161 + ci)
    scale = 1.0 / math.sqrt(D)
    PK = _randn((P, L, Hkv, plen, D), g, dt)
    PV = _randn((P, L, Hkv, plen, D), g, dt)
    K = _randn((S, L, Hkv, scap, D), g, dt)
    V = _randn((S, L, Hkv, scap, D), g, dt)
    lens = torch.randint(1, scap + 1, (S,), generator=g, dtype=torch.int32)
    lens[0] = 1
    lens[-1] = scap
    q = _randn((S, L, Hq, D), g, dt)
    kn = _randn((S, L, Hkv, D), g, dt)
    vn = _randn((S, L, Hkv, D), g, dt)
    prefix = k.Prefix(PK.to(DEV), PV.to(DEV))
    ca, cb = (k.Cache(K.to(DEV), V.to(DEV), None) for _ in range(2))
    nws = k.decode_attn_workspace_size(ca, prefix, Hq)
    wsa = torch.full((max(nws, 16) // 4,), float("nan"), device=DEV)
    wsb = torch.full((max(nws, 16) // 4,), float("nan"), device=DEV)
    oa = torch.empty((S, L, Hq, D), dtype=dt, device=DEV)
    ob = torch.empty_like(oa)
    lent = lens.to(DEV)
    k.decode_attn(ca, lent, q.to(DEV), oa, scale, k_new=kn.to(DEV), v_new=vn.to(DEV), prefix=prefix, workspace=wsa)
    xs = [_logits(R, V_, ld, ldt, kind, 91 + j) for j, (R, V_, ld, kind, det) in enumerate(specs)]
    sets = [k.LogitSet(x.to(DEV), torch.full((x.shape[0],), float("nan"), device=DEV), V_, 1.0,
                       k.Detector.zeros(x.shape[0], window=12, guard=0, tau=5.0, device=DEV) if det else None)
            for x, (R, V_, ld, kind, det) in zip(xs, specs)]
    smp = k.Sampler(*smp_args) if smp_args else None
    if smp is None:
        k.decode_attn_entropy(cb, lent, q.to(DEV), ob, scale, sets, k_new=kn.to(DEV), v_new=vn.to(DEV),
                              prefix=prefix, workspace=wsb)
    else:
        toks = [torch.full((x.shape[0],), -7, dtype=torch.int32, device=DEV) for x in xs]
        k.decode_attn_entropy_sample(cb, lent, q.to(DEV), ob, scale, sets, smp, toks, k_new=kn.to(DEV),
                                     v_new=vn.to(DEV), prefix=prefix, workspace=wsb)
    torch.cuda.synchronize()
    Kh, Vh = K.clone(), V.clone()
    for s in range(S):
        n = int(lens[s])
        Kh[s, :, :, n - 1] = kn[s]
        Vh[s, :, :, n - 1] = vn[s]
    ref, _ = oracle.decode_attn(host(Kh), host(Vh), lens.numpy(), host(q), scale,
                                prefix_K=host(PK), prefix_V=host(PV), want_psum=False)
    tol = 2e-2 if dt == torch.bfloat16 else 1e-5
    ea, eb = rowwise_rel_err(as_f64(oa), ref).max(), rowwise_rel_err(as_f64(ob), ref).max()
    say("  attention rel err: kvr_decode_attn %.2e, fused %.2e" % (ea, eb))
    assert eb <= tol
    bits = (lambda t: t.cpu().view(torch.int16)) if dt == torch.bfloat16 else (lambda t: t.cpu())
    for t in ("k", "v"):
        assert torch.equal(bits(getattr(ca, t)), bits(getattr(cb, t)))
    for j, (x, (R, V_, ld, kind, det)) in enumerate(zip(xs, specs)):
        href = oracle.entropy(host(x), V=V_)
        d = np.abs(sets[j].H.cpu().double().numpy() - href).max()
        say("  set", j, "rows", R, "H err", d)
        assert d <= 1e-4
        if det:
            od = oracle.Detector(R, window=12, guard=0, tau=5.0)
            fref = od.step(href)
            assert sets[j].detector.cnt.cpu().numpy().tolist() == [1] * R
            f = sets[j].detector.flag.cpu().numpy()
            assert ((f == fref) | (np.abs(href - 5.0) < 1e-4)).all()
        if smp is not None:
            got = toks[j].cpu().numpy()
            H = torch.empty(R, device=DEV)
            ref_tok = torch.full((R,), -7, dtype=torch.int32, device=DEV)
            ws = torch.empty(max(k.logit_entropy_sample_workspace_size(R, V_, smp.top_k), 16) // 4 + 4, device=DEV)
            k.logit_entropy_sample(x.to(DEV), H, ref_tok, smp, V=V_, workspace=ws)
            torch.cuda.synchronize()
            assert (got == ref_tok.cpu().numpy()).all(), (j, got, ref_tok.cpu().numpy())
            exact, loose = _check_tokens(host(x), V_, smp, got)
            say("  set", j, "tokens oracle-exact", exact, "near-threshold", loose)
