"""Benchmark of the KV-Rescue candidate-decode hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A step is one pass of the whole hot path over every candidate of the
workload: base decode attention over the evicted cache with the streamed
window score, top-B eviction when the cache overflows, helper decode attention
over the full context, and full-vocabulary entropy with the detector. The
default workload is the 7B-shaped base (16 problems x 8 candidates, B=64)
interleaved with the 1.5B-shaped helper over 16 shared 8192-token contexts,
with entropy over both models' logits; the 7B B=128 and 72B workloads are run
after it and reported under "workloads".

Inputs are synthetic and seeded, resident in HBM before timing starts. The
prompt is decoded (teacher-forced) before timing; then W warmup steps, then
exactly K timed steps between two synchronisations. A second, instrumented
pass of K more steps brackets every library call with timing events to get
per-call durations for the roofline. One JSON line is printed.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2608_15797_amd import accounting as acc  # noqa: E402
from paper_2608_15797_amd.profsum import source_hash  # noqa: E402
from paper_2608_15797_amd.workloads import WORKLOADS  # noqa: E402

PEAK_HBM_GBPS = 8000.0
METRIC = "candidate decode steps/s (attn+evict+entropy)"
DEFAULT_EXTRA = ("base7b", "base72b_helper", "helper4k")
def log(*a):
    print(*a, file=sys.stderr, flush=True)


def step_bytes(wl, dec, i, moved_rows=None):
    """Algorithmic bytes of decode step i by call name. moved_rows: kept rows
    per head that change slot at an eviction, on average (None = all B, the
    upper bound)."""
    out = {}
    if wl.base:
        b = wl.base
        n = dec.blen_host[dec.T_prompt + i]
        out["base_attn"] = acc.base_attn_bytes(wl, n)
        if n > b.B + b.buffer:
            out["evict"] = acc.evict_bytes(wl, n, moved_rows)
    if wl.helper:
        out["helper_attn"] = acc.helper_attn_bytes(wl, dec.hlen_host[i])
    if wl.logits:
        out["entropy"] = acc.entropy_bytes(wl)  # every logit set, one batched call
    return out


def run_workload(name, steps, warmup, instrument=True):
    from paper_2608_15797_amd.pipeline import Decoder
    base_wl = WORKLOADS[name]
    steps = steps or base_wl.steps
    wl = base_wl.with_(steps=warmup + (2 if instrument else 1) * steps)
    t0 = time.time()
    dec = Decoder(wl, device="cuda")
    torch.cuda.synchronize()
    log("[%s] buffers + input pool (%d draws) ready in %.1fs" % (name, len(dec.pool), time.time() - t0))
    dec.prompt()
    for i in range(warmup):
        dec.step(i)
    torch.cuda.synchronize()
    log("[%s] prompt (%d tokens) + %d warmup steps done" % (name, dec.T_prompt, warmup))

    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(warmup, warmup + steps):
        dec.step(i)
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end)
    log("[%s] timed %d steps: %.3f ms/step" % (name, steps, ms / steps))

    calls = {}
    moved_rows = None
    if instrument:
        # Per-call durations from event pairs around every call. The kept sets
        # of each eviction are read back after it (outside the event pairs) to
        # count the rows that changed slot: eviction's algorithmic bytes.
        timers, moved = {}, []
        for i in range(warmup + steps, warmup + 2 * steps):
            dec.step(i, timers=timers, evict_log=moved)
        torch.cuda.synchronize()
        if moved:
            b = wl.base
            moved_rows = sum(moved) / len(moved) / (b.S * b.L * b.Hkv)
        ibytes, ubound = {}, {}
        for i in range(warmup + steps, warmup + 2 * steps):
            for k, v in step_bytes(wl, dec, i, moved_rows).items():
                ibytes[k] = ibytes.get(k, 0) + v
            for k, v in step_bytes(wl, dec, i).items():
                ubound[k] = ubound.get(k, 0) + v
        for k, ev in timers.items():
            dur = [s.elapsed_time(e) for s, e in ev]
            n = len(dur)
            avg_ms = sum(dur) / n
            b_per = ibytes[k] / n
            calls[k] = dict(launches=n, avg_us=round(avg_ms * 1e3, 2),
                            bytes_per_call=int(b_per),
                            GBps=round(b_per / (avg_ms * 1e-3) / 1e9, 1),
                            frac=round(b_per / (avg_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4))
            if k == "evict":
                ub = ubound[k] / n
                calls[k].update(moved_rows_per_head=round(moved_rows, 2), bytes_upper_bound=int(ub),
                                frac_upper_bound=round(ub / (avg_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4))
        log("[%s] per-call: %s" % (name, json.dumps(calls)))

    # Whole-step algorithmic bytes of the timed window (eviction at the moved
    # rows measured above, else at the upper bound).
    total = {}
    for i in range(warmup, warmup + steps):
        for k, v in step_bytes(wl, dec, i, moved_rows).items():
            total[k] = total.get(k, 0) + v
    all_bytes = sum(total.values())

    S = (wl.base.S if wl.base else 0) + (wl.helper.S if wl.helper else 0)
    res = dict(workload=name, steps=steps, ms_per_step=ms / steps,
               steps_per_s=steps / (ms * 1e-3), cand_tokens_per_s=S * steps / (ms * 1e-3),
               alg_bytes_per_step=all_bytes / steps,
               hbm_GBps=all_bytes / (ms * 1e-3) / 1e9,
               hbm_frac=all_bytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, calls=calls)
    return res, dec, wl


def copy_bandwidth(nbytes=1 << 30):
    """Read+write bandwidth of a plain device-to-device copy of nbytes (a
    measured reference beside the 8 TB/s nameplate)."""
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    reps = 5
    dst.copy_(src)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(reps):
        dst.copy_(src)
    e.record()
    torch.cuda.synchronize()
    gbps = 2 * nbytes * reps / (s.elapsed_time(e) * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return round(gbps, 1)


def calibration_copy(nbytes=1 << 30):
    """Three dispatches of a copy kernel of known traffic (nbytes read and
    nbytes written each): a bf16 -> fp16 conversion, which runs as a kernel
    (a same-type copy may go to a DMA engine that counters do not see). Profiler
    byte counters on it calibrate those on the library's kernels."""
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda").fill_(1.0)
    dst = torch.empty(nbytes // 2, dtype=torch.float16, device="cuda")
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    torch.cuda.empty_cache()


def sampler_cost(dec, wl, reps=50):
    """Per-call time of the entropy pass alone and with the fused sampler
    (temperature 0.8, top-k 20, top-p 0.95) on the workload's logit sets."""
    from paper_2608_15797_amd import kvr
    si = dec.inputs(dec.T_prompt)
    out = {}
    for w, (lg, ls) in enumerate(zip(si.logits, wl.logits)):
        H = torch.empty(ls.R, device="cuda")
        tok = torch.empty(ls.R, dtype=torch.int32, device="cuda")
        smp = kvr.Sampler(seed=2608)
        n = kvr.logit_entropy_sample_workspace_size(ls.R, ls.V, smp.top_k)
        ws = torch.empty(max(n, 16) // 4 + 4, device="cuda")

        def ent():
            kvr.logit_entropy(lg, H, V=ls.V, workspace=dec.ews[w])

        def ent_sample():
            kvr.logit_entropy_sample(lg, H, tok, smp, V=ls.V, workspace=ws)

        res = {}
        for name, fn in (("entropy_us", ent), ("entropy_sample_us", ent_sample)):
            fn()
            torch.cuda.synchronize()
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s.record()
            for _ in range(reps):
                fn()
            e.record()
            torch.cuda.synchronize()
            res[name] = round(s.elapsed_time(e) * 1e3 / reps, 2)
        res["R"], res["V"] = ls.R, ls.V
        out["logits%d" % w] = res
    return out


def describe(wl):
    d = {"workload": wl.name, "dtype": wl.dtype}
    if wl.base:
        b = wl.base
        d["base"] = dict(S=b.S, L=b.L, Hq=b.Hq, Hkv=b.Hkv, D=b.D, B=b.B, W=b.W, buffer=b.buffer,
                         prompt=b.prompt)
    if wl.helper:
        h = wl.helper
        d["helper"] = dict(S=h.S, L=h.L, Hq=h.Hq, Hkv=h.Hkv, D=h.D, P=h.P, plen=h.plen, suffix=h.scap)
    d["logits"] = [dict(R=ls.R, V=ls.V) for ls in wl.logits]
    return d


def traffic_record(name, call):
    """The traffic record of `call` (profiles/traffic_<workload>.json, written
    by profsum --traffic from rocprofv3 PMC counters), or None when it is
    missing or was taken on other kernel sources."""
    path = os.path.join(ROOT, "profiles", "traffic_%s.json" % name)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    rec = t.get("calls", {}).get(call)
    if rec is None or rec.get("source_hash") != source_hash(call):
        return None
    return rec


def traffic_for(name, call):
    """Measured HBM bytes per call of `call`, or None (see traffic_record)."""
    rec = traffic_record(name, call)
    return None if rec is None else rec["bytes_per_call"]


def attach_traffic(name, calls):
    """Add the measured HBM bytes per call to every call that has a current
    traffic record, with their ratio to the algorithmic bytes of the same
    dispatches (the counter run's own, prompt included) when the record
    holds them."""
    for call, c in calls.items():
        rec = traffic_record(name, call)
        if rec is not None:
            c["measured_bytes_per_call"] = int(rec["bytes_per_call"])
            if "measured_over_alg" in rec:
                c["measured_over_alg"] = rec["measured_over_alg"]


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(dec, wl, min_s=10.0):
    """The fp64 oracle timed on this host with all its OpenMP threads and
    with one thread (a reported baseline, not a target); see
    oracle_sample for the sample. `value` is the all-threads rate."""
    import oracle
    n_all = oracle.threads()
    steps, secs, desc, done, problems = oracle_sample(dec, wl, min_s)
    oracle.set_threads(1)
    try:
        steps1, secs1, _, done1, _ = oracle_sample(dec, wl, min_s)
    finally:
        oracle.set_threads(n_all)
    return dict(value=round(steps / secs, 6), unit="steps/s", cores=n_all, kind="oracle",
                single_thread_value=round(steps1 / secs1, 6), nproc=os.cpu_count(), cpu_model=cpu_model(),
                sample="%d problem-steps of %d problems per step (%s), %.1f s of oracle time on %d threads; "
                       "%d problem-steps, %.1f s on one thread"
                % (done, problems, "; ".join(desc), secs, n_all, done1, secs1))


def oracle_sample(dec, wl, min_s):
    """One problem's share of a decode step (its candidates' base attention,
    helper attention and logit rows) at a time, problem after problem and
    step after step, until at least `min_s` seconds of oracle time. Returns
    (whole steps, seconds, description, problem-steps, problems per step).
    Host copies are made outside the timing."""
    import numpy as np

    import oracle

    def host(t):
        t = t.detach().cpu().contiguous()
        return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()

    b, h = wl.base, wl.helper
    problems = 8 if wl.name == "base72b_helper" else 16
    secs, done = 0.0, 0
    desc = []
    for i in range(wl.steps):
        t = dec.T_prompt + i
        si = dec.inputs(t)
        for p in range(problems):
            if b:
                nb = b.S // problems
                sl = slice(p * nb, (p + 1) * nb)
                n = dec.blen_host[t]
                K, V, q = host(dec.bcache.k[sl]), host(dec.bcache.v[sl]), host(si.bq[sl])
                t0 = time.perf_counter()
                oracle.decode_attn(K, V, n, q, dec.bscale)
                secs += time.perf_counter() - t0
                if done == 0:
                    desc.append("base %d of %d sequences" % (nb, b.S))
            if h:
                nh = h.S // problems
                sl = slice(p * nh, (p + 1) * nh)
                C = h.S // h.P
                psl = slice((p * nh) // C, max((p * nh) // C + 1, ((p + 1) * nh) // C))
                u = dec.hlen_host[i]
                PK, PV = host(dec.prefix.k[psl]), host(dec.prefix.v[psl])
                K, V, q = host(dec.hcache.k[sl]), host(dec.hcache.v[sl]), host(si.hq[sl])
                t0 = time.perf_counter()
                oracle.decode_attn(K, V, u, q, h.softmax_scale, prefix_K=PK, prefix_V=PV,
                                   want_psum=False)
                secs += time.perf_counter() - t0
                if done == 0:
                    desc.append("helper %d of %d candidates over context %d" % (nh, h.S, h.plen))
            for w, ls in enumerate(wl.logits):
                nr = max(1, ls.R // problems)
                x = host(si.logits[w][p * nr:(p + 1) * nr])
                t0 = time.perf_counter()
                oracle.entropy(x, V=ls.V)
                secs += time.perf_counter() - t0
                if done == 0:
                    desc.append("entropy %d of %d rows (V=%d)" % (nr, ls.R, ls.V))
            done += 1
            if secs >= min_s:
                break
        if secs >= min_s:
            break
    return done / problems, secs, desc, done, problems


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=0, help="timed steps (default: the workload's decode steps)")
    ap.add_argument("--warmup", type=int, default=32)
    ap.add_argument("--workload", default="base7b_helper", choices=sorted(WORKLOADS))
    ap.add_argument("--extra", default=",".join(DEFAULT_EXTRA),
                    help="comma-separated workloads also reported (empty: none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-instrument", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a 1 GiB copy kernel three times (the known-size reference "
                         "that scales rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_calibration:
        calibration_copy()
    copy_ref = copy_bandwidth()

    res, dec, wl = run_workload(args.workload, args.steps, args.warmup, not args.no_instrument)
    steps = res["steps"]
    calls = res["calls"]
    attach_traffic(args.workload, calls)
    roof = None
    if calls:
        dom = max(calls, key=lambda k: calls[k]["bytes_per_call"] * calls[k]["launches"])
        c = calls[dom]
        roof = dict(bound="hbm", achieved=c["GBps"], peak=PEAK_HBM_GBPS, unit="GB/s", frac=c["frac"],
                    traffic=traffic_for(args.workload, dom), call=dom,
                    alg_bytes_per_call=c["bytes_per_call"], avg_us=c["avg_us"])
    sampler = sampler_cost(dec, wl) if not args.no_instrument else None
    if sampler:
        log("[%s] sampler: %s" % (args.workload, json.dumps(sampler)))
    cpu = None
    if not args.no_cpu_baseline:
        t0 = time.time()
        cpu = cpu_baseline(dec, wl)
        log("[cpu baseline] %.1fs: %s" % (time.time() - t0, json.dumps(cpu)))
    del dec
    torch.cuda.empty_cache()

    extra = {}
    for name in [x for x in args.extra.split(",") if x and x != args.workload]:
        r, d, _ = run_workload(name, 0, args.warmup, not args.no_instrument)
        attach_traffic(name, r["calls"])
        del d
        torch.cuda.empty_cache()
        extra[name] = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in r.items()}

    cfg = describe(WORKLOADS[args.workload])
    cfg.update(cand_tokens_per_s=round(res["cand_tokens_per_s"], 1),
               alg_bytes_per_step=int(res["alg_bytes_per_step"]),
               hbm_GBps=round(res["hbm_GBps"], 1), hbm_frac_of_peak=round(res["hbm_frac"], 4),
               calls=calls)
    line = {
        "metric": METRIC, "value": round(res["steps_per_s"], 3), "unit": "steps/s",
        "n_gpus": 1, "steps": steps, "warmup": args.warmup,
        "ms_per_step": round(res["ms_per_step"], 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded, Qwen2.5-Math shapes)",
        "config": cfg, "roofline": roof, "cpu_baseline": cpu, "workloads": extra,
        "sampler": sampler,
        "copy_ref_GBps": copy_ref,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
