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


def _mutable(dec):
    """Every buffer a decode step writes."""
    ts = [dec.bcache.k, dec.bcache.v, dec.bcache.pos, dec.scores, dec.kept, dec.bout,
          dec.hcache.k, dec.hcache.v, dec.hout, dec.hws,
          dec.detector.hist, dec.detector.cnt, dec.detector.flag, *dec.H]
    return [t for t in ts if t is not None]


def _same(a, b):
    if a.dtype == torch.bfloat16:
        return torch.equal(a.view(torch.int16), b.view(torch.int16))
    return torch.equal(a, b)


def test_decode_cycle_with_evictions_graph_replays_match_eager():
    """40 decode steps holding two evictions and their observation windows,
    captured as one HIP graph: from the same starting state, every replay
    leaves every buffer the steps write (caches, positions, scores, kept
    sets, outputs, entropies, detector) bit for bit as the eager steps do."""
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_15797_amd.pipeline import Decoder
    from paper_2608_15797_amd.workloads import BaseShape, HelperShape, LogitSet, Workload
    wl = Workload(name="graph_cycle", dtype="bf16", steps=80,
                  base=BaseShape(S=8, L=2, Hq=28, Hkv=4, D=128, B=16, W=8, buffer=16, prompt=32),
                  helper=HelperShape(S=8, L=2, Hq=12, Hkv=2, D=128, P=8, plen=700),
                  logits=(LogitSet(R=8, V=152064, std=3.0, n_boost=5, boost=10.0),
                          LogitSet(R=8, V=151936, std=1.0)),
                  detector=(12, 3, 7.0), seed=78)
    dec = Decoder(wl, device="cuda")
    dec.prompt()
    i0, K = 6, 40
    for i in range(i0):
        dec.step(i)
    b = wl.base
    steps = list(range(i0, i0 + K))
    ev = [i for i in steps if dec.blen_host[dec.T_prompt + i] > b.B + b.buffer]
    say("graph cycle: steps", steps[0], "-", steps[-1], "evictions at", ev)
    assert len(ev) == 2
    torch.cuda.synchronize()
    start = [t.clone() for t in _mutable(dec)]

    def restore():
        for t, s in zip(_mutable(dec), start):
            t.copy_(s)
        torch.cuda.synchronize()

    for i in steps:
        dec.step(i)
    torch.cuda.synchronize()
    eager = [t.clone() for t in _mutable(dec)]
    assert not all(_same(a, s) for a, s in zip(eager, start))

    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    restore()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        dec.step(steps[0])  # warm the launch path on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        for i in steps:
            dec.step(i)
    torch.cuda.synchronize()
    for rep in range(2):
        restore()
        torch.randn(1 << 20, device="cuda").sum()  # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for j, (a, r) in enumerate(zip(_mutable(dec), eager)):
            assert _same(a, r), (rep, j)
