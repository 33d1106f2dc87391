"""Program for the HBM byte-counter passes of the attention and eviction calls.

    python -m paper_2608_15797_amd.trafficrun [--workload NAME] [--steps N]

Runs a calibration copy (three dispatches of a 1 GiB bf16 -> fp16 conversion:
1 GiB read and 1 GiB written each, the reference that profsum scales the
FETCH_SIZE / WRITE_SIZE counters by), then the workload's prompt and N decode
steps of the whole hot path: base attention (with its evictions), helper
attention and the batched logit-entropy call.
Run it under one `rocprofv3 --pmc FETCH_SIZE` and one `--pmc WRITE_SIZE` pass
and give both result directories to `profsum --traffic`. N defaults to the
workload's decode steps, the benchmark's timed window, so the per-dispatch
averages cover the same mix of cache and suffix lengths (the prompt adds the
same few hundred dispatches as in the benchmark's own run).

The last line printed is a JSON object with the algorithmic bytes per
dispatch of every call over exactly the dispatches of this run (prompt
included; eviction at the kept rows that changed slot, read back from each
eviction's kept set), to set against the measured bytes per dispatch.
"""
from __future__ import annotations

import argparse
import sys
import time

import torch


def calibration_copy(nbytes: int = 1 << 30) -> None:
    # A conversion runs as a kernel; a same-type copy may go to a DMA engine
    # that the counters do not see.
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda").fill_(1.0)
    dst = torch.empty(nbytes // 2, dtype=torch.float16, device="cuda")
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    torch.cuda.empty_cache()


def main(argv=None) -> None:
    import json

    from paper_2608_15797_amd import accounting as acc
    from paper_2608_15797_amd.pipeline import Decoder
    from paper_2608_15797_amd.workloads import WORKLOADS

    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--workload", default="base7b_helper", choices=sorted(WORKLOADS))
    ap.add_argument("--steps", type=int, default=0, help="decode steps (default: the workload's)")
    args = ap.parse_args(argv)
    calibration_copy()
    print("calibration copy done", flush=True)
    wl = WORKLOADS[args.workload]
    if args.steps:
        wl = wl.with_(steps=args.steps)
    t0 = time.time()
    dec = Decoder(wl, device="cuda")
    alg = {}  # call -> [bytes, dispatches]

    def count(call, nbytes):
        a = alg.setdefault(call, [0, 0])
        a[0] += nbytes
        a[1] += 1

    def base(t, si):
        moved = []
        if dec.base_token(t, si, evict_log=moved):
            b = wl.base
            count("evict", acc.evict_bytes(wl, dec.blen_host[t], moved[0] / (b.S * b.L * b.Hkv)))
        count("base_attn", acc.base_attn_bytes(wl, dec.blen_host[t]))

    for t in range(dec.T_prompt):
        base(t, dec.inputs(t))
    torch.cuda.synchronize()
    print("[%s] prompt (%d tokens) done" % (wl.name, dec.T_prompt), flush=True)
    for i in range(wl.steps):
        t = dec.T_prompt + i
        si = dec.inputs(t)
        if wl.base:
            base(t, si)
        if wl.helper:
            dec.helper_token(i, si)
            count("helper_attn", acc.helper_attn_bytes(wl, dec.hlen_host[i]))
        if wl.logits:
            dec.entropy(si)
            count("entropy", acc.entropy_bytes(wl))
        if (i + 1) % 512 == 0:
            torch.cuda.synchronize()
            print("[%s] %d steps (%.1fs)" % (wl.name, i + 1, time.time() - t0), flush=True)
    torch.cuda.synchronize()
    print("done", flush=True)
    print(json.dumps({"workload": wl.name, "alg_bytes_per_dispatch": {k: int(round(v[0] / v[1])) for k, v in alg.items()},
                      "dispatches": {k: v[1] for k, v in alg.items()}}), flush=True)


if __name__ == "__main__":
    sys.exit(main())
