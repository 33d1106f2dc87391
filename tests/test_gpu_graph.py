"""One whole decode step of a base + helper workload (base attention with both
models' entropy rows in one launch, then the helper's context and suffix
kernels) captured in a HIP graph and replayed: the library allocates nothing
and clears nothing with memsets on this path, so the step can be captured.
Every replay, with eager work and synchronisations between replays, must give
bit for bit the eager step's outputs and entropies; the detector counts one
push per replay."""
import pytest
import torch

from gpu_util import say

pytestmark = pytest.mark.gpu


def test_decode_step_graph_replays_match_eager():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_15797_amd.pipeline import Decoder
    from paper_2608_15797_amd.workloads import BaseShape, HelperShape, LogitSet, Workload
    wl = Workload(name="graph_small", dtype="bf16", steps=16,
                  base=BaseShape(S=8, L=2, Hq=28, Hkv=4, D=128, B=64, W=32, buffer=64, prompt=32),
                  helper=HelperShape(S=8, L=2, Hq=12, Hkv=2, D=128, P=2, plen=1000),
                  logits=(LogitSet(R=8, V=152064, std=3.0, n_boost=5, boost=10.0),
                          LogitSet(R=8, V=151936, std=1.0)),
                  seed=77)
    dec = Decoder(wl, device="cuda")
    dec.prompt()
    step = 10
    for i in range(step):
        dec.step(i)
    b = wl.base
    n = dec.blen_host[dec.T_prompt + step]
    # Before the observation window and far from an eviction: the step's
    # appends rewrite the same slots, so repeating it is idempotent.
    assert n < b.B + b.buffer + 2 - b.W
    say("graph step", step, "base n", n, "helper suffix", dec.hlen_host[step])
    dec.step(step)
    torch.cuda.synchronize()
    ref = [dec.bout.clone(), dec.hout.clone()] + [h.clone() for h in dec.H]
    cnt0 = dec.detector.cnt.clone()

    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        dec.step(step)  # warm the launch path on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        dec.step(step)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (dec.bout, dec.hout, *dec.H):
            t.fill_(0)
        torch.randn(1 << 20, device="cuda").sum()  # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = [dec.bout, dec.hout] + list(dec.H)
        for j, (a, r) in enumerate(zip(got, ref)):
            same = torch.equal(a.view(torch.int16), r.view(torch.int16)) if a.dtype == torch.bfloat16 \
                else torch.equal(a, r)
            assert same, (rep, j)
    # Eager, side-stream warm-up and three replays after the reference step.
    assert torch.equal(dec.detector.cnt, cnt0 + 4)
