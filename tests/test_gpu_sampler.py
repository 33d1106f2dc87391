"""GPU parity of kvr_logit_entropy_sample (entropy of Eq. (4), the detector and
the fused temperature / top-k / top-p sampler) against oracle/sampler.py and
the entropy oracle, through the C ABI.

Tokens: the sampled id equals the oracle's wherever the oracle's fp64
decisions sit at least 1e-5 (in probability mass) from their thresholds (the
top-p cut and the inverse-CDF step); closer than that the GPU's float32 sums
may take either side, so the GPU token must then be a member of the oracle's
top-k, at most one position from the oracle's pick in the sorted order.
Entropy within 1e-4 absolute; detector state equal.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import host, say
from oracle import sampler as osamp

pytestmark = pytest.mark.gpu

DEV = "cuda"
MARGIN = 1e-5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_15797_amd import kvr  # noqa: F401  (fails loudly if libkvr.so is missing)
    yield


def kvr():
    from paper_2608_15797_amd import kvr as k
    return k


def _logits(R, V, ld, dtype, kind, seed):
    from paper_2608_15797_amd import synth
    g = torch.Generator().manual_seed(seed)
    if kind == "boosted":
        x = synth.boosted_logits(R, V, 3.0, 5, 10.0, seed, device="cpu", dtype=torch.float32)
    elif kind == "ties":
        x = torch.randint(-4, 3, (R, V), generator=g).float()
    elif kind == "flat":
        x = torch.randn((R, V), generator=g) * 0.1
    else:
        x = torch.randn((R, V), generator=g) * float(kind)
    out = torch.zeros((R, ld), dtype=dtype)
    out[:, :V] = x.to(dtype)
    return out


def _run(logits, V, smp, det=None):
    k = kvr()
    R = logits.shape[0]
    H = torch.empty(R, device=DEV)
    tok = torch.full((R,), -7, dtype=torch.int32, device=DEV)
    ws_n = k.logit_entropy_sample_workspace_size(R, V, smp.top_k)
    ws = torch.empty(max(ws_n, 16) // 4 + 4, device=DEV)
    k.logit_entropy_sample(logits, H, tok, smp, V=V, detector=det, workspace=ws)
    torch.cuda.synchronize()
    return H.cpu().double().numpy(), tok.cpu().numpy()


def _check_tokens(x_host, V, smp, got):
    exact = loose = 0
    for r in range(x_host.shape[0]):
        u = osamp.uniform(smp.seed, smp.step, r)
        t, d = osamp.sample_row(x_host[r], V, smp.temperature, smp.top_k, smp.top_p, u)
        if min(d["margin_u"], d["margin_p"]) >= MARGIN:
            assert got[r] == t, (r, got[r], t, d["margin_u"], d["margin_p"])
            exact += 1
        else:
            order = d["order"].tolist()
            assert got[r] in order, (r, got[r])
            assert abs(order.index(int(got[r])) - d["pick"]) <= 1, (r, got[r], t)
            loose += 1
    return exact, loose


CASES = [
    # R, V, ld, dtype, logits, top_k, top_p, temperature
    (3, 7, 7, torch.float32, "2.0", 20, 0.95, 0.8),            # V < top_k, scalar loads
    (4, 1024, 1024, torch.float32, "2.0", 20, 0.95, 0.8),
    (5, 1000, 1003, torch.bfloat16, "3.0", 20, 0.95, 0.8),     # odd ld: scalar path
    (6, 4099, 4104, torch.bfloat16, "boosted", 20, 0.95, 0.8),  # V % 8 tail
    (8, 151936, 151936, torch.bfloat16, "boosted", 20, 0.95, 0.8),
    (16, 32000, 32000, torch.float32, "1.0", 64, 1.0, 1.0),    # largest k, no nucleus cut
    (16, 32000, 32000, torch.bfloat16, "1.0", 1, 0.95, 0.8),   # greedy
    (4, 5000, 5008, torch.bfloat16, "flat", 20, 0.95, 0.8),    # near-uniform probabilities
    # Many exactly equal logits: the top 20 all share the largest value, so the
    # kept tokens are the 19 lowest ids holding it (top_p 0.93 lies between the
    # equal-probability cumulative steps 0.90 and 0.95).
    (6, 4096, 4096, torch.bfloat16, "ties", 20, 0.93, 0.8),
    (2, 300000, 300000, torch.bfloat16, "boosted", 7, 0.5, 0.6),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "R%dV%dld%d_%s_%s_k%d_p%g" % (
    c[0], c[1], c[2], str(c[3]).split(".")[-1], c[4], c[5], c[6]))
def test_sampler_parity(case):
    R, V, ld, dt, kind, top_k, top_p, T = case
    k = kvr()
    x = _logits(R, V, ld, dt, kind, seed=R * 7 + V)
    xd = x.to(DEV)
    xh = host(x)
    Href = oracle.entropy(xh, V=V)
    tot_exact = tot_loose = 0
    for step in (0, 1, 12345):
        smp = k.Sampler(temperature=T, top_k=top_k, top_p=top_p, seed=0xC0FFEE + R, step=step)
        H, tok = _run(xd, V, smp)
        assert np.abs(H - Href).max() <= 1e-4
        e, l_ = _check_tokens(xh, V, smp, tok)
        tot_exact += e
        tot_loose += l_
    say("  tokens: %d exact, %d within the rounding margin" % (tot_exact, tot_loose))
    assert tot_exact >= tot_loose


def test_sampler_workload_rows_full_size():
    """The 7B workload's logit shape (128 rows x 152064, bf16, five boosted
    tokens per row): every row checked at several steps."""
    k = kvr()
    R, V = 128, 152064
    x = _logits(R, V, V, torch.bfloat16, "boosted", seed=31)
    xd, xh = x.to(DEV), host(x)
    for step in (0, 7, 4095):
        smp = k.Sampler(seed=2608, step=step)
        H, tok = _run(xd, V, smp)
        e, l_ = _check_tokens(xh, V, smp, tok)
        say("  step %d: %d exact, %d within margin" % (step, e, l_))
    assert np.abs(H - oracle.entropy(xh, V=V)).max() <= 1e-4


def test_sampler_detector_state():
    """The detector runs in the sampling merge exactly as in kvr_logit_entropy."""
    k = kvr()
    R, V = 5, 2048
    det = k.Detector.zeros(R, window=3, guard=4, tau=5.0)
    ref = oracle.Detector(R, window=3, guard=4, tau=5.0)
    for i in range(8):
        x = _logits(R, V, V, torch.float32, "flat" if i % 2 else "2.0", seed=100 + i)
        H, _ = _run(x.to(DEV), V, k.Sampler(step=i), det)
        ref.step(oracle.entropy(host(x), V=V))
    np.testing.assert_allclose(det.hist.cpu().numpy(), ref.hist, atol=1e-4)
    assert np.array_equal(det.cnt.cpu().numpy(), ref.cnt)
    assert np.array_equal(det.flag.cpu().numpy(), ref.flag)


def test_sampler_rejects_bad_settings():
    k = kvr()
    x = torch.zeros((2, 64), device=DEV)
    H = torch.empty(2, device=DEV)
    tok = torch.empty(2, dtype=torch.int32, device=DEV)
    ws = torch.empty(4096, device=DEV)
    for smp in (k.Sampler(temperature=0.0), k.Sampler(top_k=0), k.Sampler(top_k=65),
                k.Sampler(top_p=0.0), k.Sampler(top_p=1.5)):
        with pytest.raises(k.KvrError):
            k.logit_entropy_sample(x, H, tok, smp, workspace=ws)
    with pytest.raises(k.KvrError):
        k.logit_entropy_sample(x, H, tok, k.Sampler(), workspace=None)
