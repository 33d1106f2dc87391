"""The allocation-free entropy entry point (kvr_logit_entropy_batch_noalloc)
against the workspace entry point (kvr_logit_entropy_batch), through the C
ABI: two calls in a row, the second on a smaller input, each compared with
the workspace call on the same rows (entropies within 1e-4 absolute, the
bar of the entropy parity tests; detector state identical) and with the
oracle. The inputs need split partials, so the library's scratch is used."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import host, say

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _sets(k, specs, seed):
    g = torch.Generator().manual_seed(seed)
    out = []
    for R, V, std in specs:
        x = (torch.randn((R, V), generator=g) * std)
        x[0, :7] = float("-inf")
        x[-1, :5] += 10.0
        out.append(x.to(torch.bfloat16))
    return out


def _run(k, xs, noalloc):
    sets = [k.LogitSet(x.to(DEV), torch.full((x.shape[0],), float("nan"), device=DEV), x.shape[1],
                       1.0, k.Detector.zeros(x.shape[0], window=12, guard=1, tau=5.0, device=DEV))
            for x in xs]
    if noalloc:
        k.logit_entropy_batch_noalloc(sets)
    else:
        need = k.logit_entropy_batch_workspace_size([tuple(x.shape) for x in xs])
        ws = torch.zeros(max(need, 16) // 4, device=DEV)
        k.logit_entropy_batch(sets, workspace=ws)
    torch.cuda.synchronize()
    return sets


def test_noalloc_matches_workspace_call_twice():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_15797_amd import kvr as k
    # First call: two logit sets of 64 rows (split partials in the scratch);
    # second call: one smaller set, so stale partials of the first call sit
    # in the scratch beyond what the second call writes.
    for call, specs in enumerate([[(64, 152064, 3.0), (64, 151936, 1.0)], [(8, 50000, 2.0)]]):
        need = k.logit_entropy_batch_workspace_size([(R, V) for R, V, _ in specs])
        assert 0 < need <= k.ENTROPY_SCRATCH_BYTES, need
        xs = _sets(k, specs, 900 + call)
        a = _run(k, xs, noalloc=True)
        b = _run(k, xs, noalloc=False)
        for j, (sa, sb, x) in enumerate(zip(a, b, xs)):
            ha, hb = sa.H.cpu().double().numpy(), sb.H.cpu().double().numpy()
            ref = oracle.entropy(host(x))
            say("call", call, "set", j, "rows", x.shape[0], "scratch bytes", need,
                "max |noalloc - workspace|", np.abs(ha - hb).max(), "max |noalloc - oracle|", np.abs(ha - ref).max())
            assert np.abs(ha - hb).max() <= 1e-4
            assert np.abs(ha - ref).max() <= 1e-4
            assert torch.equal(sa.detector.hist.cpu(), sb.detector.hist.cpu())
            assert torch.equal(sa.detector.cnt.cpu(), sb.detector.cnt.cpu())
            assert torch.equal(sa.detector.flag.cpu(), sb.detector.flag.cpu())
