"""Per-layer launches of base decode attention: eager and as a HIP graph.

    python -m paper_2608_15797_amd.layerbench [--workload NAME] [--reps N]

A model decodes one layer at a time (layer l + 1's queries need layer l's
output), while the decode benchmark batches the L layers of a step into one
launch per call, since its synthetic queries are all known up front. This
program times the per-layer alternative on the same base shape: L calls of
kvr_decode_attn per step on L single-layer caches (one tensor per layer, as a
model keeps them), issued eagerly and as one captured HIP graph per step, next
to the layer-batched call. Every live length is the mean of the eviction
cycle, B + (buffer + 2) / 2, and the new token is appended as in decode (the
same slot each repetition). Before timing, the per-layer outputs are checked
bit for bit against the batched call's (the kernel computes each (sequence,
layer, KV head) unit the same way in both), and three graph replays, with
eager launches and synchronisations between them, against the eager ones.
Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import math

import torch

from paper_2608_15797_amd import kvr, synth
from paper_2608_15797_amd.workloads import WORKLOADS


def _time(fn, reps: int) -> float:
    fn()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        fn()
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) * 1000.0 / reps


def run(workload: str = "base7b_helper", reps: int = 200, seed: int = 11, base=None) -> dict:
    """`base` (a workloads.BaseShape) overrides the workload's base shape."""
    b = base if base is not None else WORKLOADS[workload].base
    if b is None:
        raise SystemExit("%s has no base model" % workload)
    dt = torch.bfloat16
    S, L, Hq, Hkv, D, cap = b.S, b.L, b.Hq, b.Hkv, b.D, b.cache_cap
    n = b.B + (b.buffer + 2) // 2
    dev = "cuda"
    K = torch.empty((S, L, Hkv, cap, D), dtype=dt, device=dev)
    V = torch.empty_like(K)
    synth.fill_normal_(K, 1.0, seed, "layers", "k")
    synth.fill_normal_(V, 1.0, seed, "layers", "v")
    q = synth.normal((S, L, Hq, D), 1.0, seed, "layers", "q", device=dev, dtype=dt)
    kn = synth.normal((S, L, Hkv, D), 1.0, seed, "layers", "kn", device=dev, dtype=dt)
    vn = synth.normal((S, L, Hkv, D), 1.0, seed, "layers", "vn", device=dev, dtype=dt)
    ln = torch.full((S,), n, dtype=torch.int32, device=dev)
    scale = 1.0 / math.sqrt(D)
    out = torch.empty((S, L, Hq, D), dtype=dt, device=dev)
    cache = kvr.Cache(K, V, None)

    # One single-layer cache (and input slices) per layer.
    lk = [K[:, l:l + 1].contiguous() for l in range(L)]
    lv = [V[:, l:l + 1].contiguous() for l in range(L)]
    lcache = [kvr.Cache(lk[l], lv[l], None) for l in range(L)]
    lq = [q[:, l:l + 1].contiguous() for l in range(L)]
    lkn = [kn[:, l:l + 1].contiguous() for l in range(L)]
    lvn = [vn[:, l:l + 1].contiguous() for l in range(L)]
    lout = [torch.empty((S, 1, Hq, D), dtype=dt, device=dev) for _ in range(L)]

    def batched():
        kvr.decode_attn(cache, ln, q, out, scale, k_new=kn, v_new=vn)

    def per_layer():
        for l in range(L):
            kvr.decode_attn(lcache[l], ln, lq[l], lout[l], scale, k_new=lkn[l], v_new=lvn[l])

    batched()
    per_layer()
    torch.cuda.synchronize()
    eager = torch.cat(lout, dim=1)
    same_as_batched = bool(torch.equal(eager.view(torch.int16), out.view(torch.int16)))

    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        per_layer()  # warm the launch path on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        per_layer()
    replays_match = True
    for _ in range(3):
        for t in lout:
            t.fill_(0)
        batched()  # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        replays_match &= bool(torch.equal(torch.cat(lout, dim=1).view(torch.int16), eager.view(torch.int16)))

    t_batched = _time(batched, reps)
    t_eager = _time(per_layer, reps)
    t_graph = _time(graph.replay, reps)
    layer_bytes = S * Hkv * n * D * 2 * 2 + S * Hq * D * 2 * 2 + S * Hkv * D * 2 * 2
    return dict(workload=workload, S=S, L=L, n=n, layer_MB=round(layer_bytes / 1e6, 2),
                layer_batched_us=round(t_batched, 2), per_layer_eager_us=round(t_eager, 2),
                per_layer_graph_us=round(t_graph, 2),
                per_layer_graph_us_per_layer=round(t_graph / L, 2),
                batched_GBps=round(layer_bytes * L / (t_batched * 1e-6) / 1e9, 1),
                per_layer_graph_GBps=round(layer_bytes * L / (t_graph * 1e-6) / 1e9, 1),
                per_layer_same_as_batched=same_as_batched, graph_replays_match=replays_match)


def main(argv=None) -> None:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--workload", default="base7b_helper", choices=sorted(w for w in WORKLOADS if WORKLOADS[w].base))
    ap.add_argument("--reps", type=int, default=200)
    args = ap.parse_args(argv)
    print(json.dumps(run(args.workload, args.reps)), flush=True)


if __name__ == "__main__":
    main()
