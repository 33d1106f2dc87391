"""Program for the HBM byte-counter passes of the attention and eviction calls.

    python -m paper_2608_15797_amd.trafficrun [--workload NAME] [--steps K] [--warmup W]

Runs a calibration copy (three dispatches of a 1 GiB bf16 -> fp16 conversion:
1 GiB read and 1 GiB written each, the reference that profsum scales the
FETCH_SIZE / WRITE_SIZE counters by), then the workload's prompt, the W warmup
steps and the K decode steps that bench.py times for the same --steps and
--warmup (same placement of the window), between two marker kernels. Run it
under one `rocprofv3 --pmc FETCH_SIZE` and one `--pmc WRITE_SIZE` pass and
give both result directories to `profsum --traffic --window 0 1`, so the
per-dispatch averages cover exactly the timed window's dispatches.

The last line printed is a JSON object with the algorithmic bytes per
dispatch of every call over exactly the window's dispatches (eviction at the
kept rows that changed slot, read back from each eviction's kept set), to set
against the measured bytes per dispatch, and the window itself.
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

    from paper_2608_15797_amd.benchplan import Schedule, cycle_steps, place_window, step_bytes, window_stats
    from paper_2608_15797_amd.pipeline import Decoder
    from paper_2608_15797_amd.workloads import WORKLOADS

    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--workload", default="base72b_helper", choices=sorted(WORKLOADS))
    ap.add_argument("--steps", type=int, default=0, help="window steps (default: one whole cycle)")
    ap.add_argument("--warmup", type=int, default=5)
    args = ap.parse_args(argv)
    calibration_copy()
    print("calibration copy done", flush=True)
    wl0 = WORKLOADS[args.workload]
    K = args.steps or cycle_steps(wl0)
    s0 = place_window(wl0, K, args.warmup)
    wl = wl0.with_(steps=s0 + K + 1)
    t0 = time.time()
    dec = Decoder(wl, device="cuda")
    alg = {}  # call -> [bytes, dispatches]

    def count(call, nbytes):
        a = alg.setdefault(call, [0, 0])
        a[0] += nbytes
        a[1] += 1

    def step(i, counted):
        moved = []
        dec.step(i, evict_log=moved)
        if counted:
            b = wl.base
            mr = moved[0] / (b.S * b.L * b.Hkv) if moved else None
            for call, nbytes in step_bytes(wl, dec, i, mr).items():
                count(call, nbytes)

    dec.prompt()
    for i in range(s0 - args.warmup, s0):
        step(i, False)
    torch.cuda.synchronize()
    print("[%s] prompt (%d tokens) + %d warmup steps done" % (wl.name, dec.T_prompt, args.warmup), flush=True)
    torch.cuda._sleep(1)
    for i in range(s0, s0 + K):
        step(i, True)
        if (i - s0 + 1) % 128 == 0:
            torch.cuda.synchronize()
            print("[%s] %d steps (%.1fs)" % (wl.name, i - s0 + 1, time.time() - t0), flush=True)
    torch.cuda._sleep(1)
    torch.cuda.synchronize()
    print("done", flush=True)
    wstat = window_stats(wl, Schedule(wl, s0 + K + 1), s0, K)
    print(json.dumps({"workload": wl.name, "window": wstat,
                      "alg_bytes_per_dispatch": {k: int(round(v[0] / v[1])) for k, v in alg.items()},
                      "dispatches": {k: v[1] for k, v in alg.items()}}), flush=True)


if __name__ == "__main__":
    sys.exit(main())
