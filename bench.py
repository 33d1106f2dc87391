"""Benchmark of the KV-Rescue candidate-decode hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A step is one pass of the whole hot path over every candidate of the
workload: base decode attention over the evicted cache with the streamed
window score, top-B eviction when the cache overflows, helper decode attention
over the full context, and full-vocabulary entropy with the detector. The
default workload is the largest: the 72B-shaped base (8 problems x 4
candidates, B=64) interleaved with the 1.5B-shaped helper over 32 private
16384-token contexts, with entropy over the base logits. The 7B + helper,
7B B=128 and 4096-token helper workloads run after it and are reported under
"workloads", each over one whole cycle timed without events between the calls
(an event pair costs a few microseconds of GPU time, up to 8% of the smaller
steps); their per-call table comes from the replay.

Placement of the timed window. Lengths and inputs are functions of the decode
step index (all candidates advance in lockstep), so the K timed steps can be
any K consecutive step indices. They are placed so that the window holds an
eviction and, before it, as many as fit of the other W_policy - 1 steps of
its observation window (the steps that stream the score), choosing among the
workload's evictions the one whose window has the mean helper suffix length
closest to the suffix cycle's mean. The W warmup
steps are the W step indices just before the window; the step indices between
the prompt and the warmup are not run. The defaults, K = 20 and W = 5, time
one eviction with its observation window; --steps 0 times one whole cycle:
whole eviction periods covering the 512-token helper suffix cycle.

Inputs are synthetic and seeded, resident in HBM before timing starts. The
prompt is decoded (teacher-forced) first; then the warmup steps, then exactly
K timed steps between two synchronisations, with HIP events on the launch
stream around each call of the dominant call (the roofline's kernel time).
A replay of the same K step indices brackets every call with events for the
per-call table. The entropies ride in the base-attention launch (in the
helper's context launch when there is no base model); a second pass runs, at
every step of the window, the fused call, the same attention call alone and
the entropy call alone, one after the other, three times: the difference
between the fused call and the attention alone is entropy's marginal time
("entropy_marginal"). Unless the window already is one, a whole
cycle is then timed and replayed the same way and reported under "cycle".

Marker kernels (torch.cuda._sleep, a one-thread spin kernel) bracket every
pass, so that a profile of this command can be cut into its passes (profsum
--window): for each workload in order, marker before the timed pass, after
it, after its replay, after the entropy-marginal pass (when entropy is fused), and,
when a cycle is run, after the cycle's timed pass and after its replay.

One JSON line is printed.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2608_15797_amd import accounting as acc  # noqa: E402
from paper_2608_15797_amd.benchplan import (PEAK_HBM_GBPS, Schedule, cycle_start, cycle_steps,  # noqa: E402
                                             dominant_call, place_window, step_bytes, window_bytes,
                                             window_stats)
from paper_2608_15797_amd.workloads import WORKLOADS  # noqa: E402

METRIC = "candidate decode steps/s (attn+evict+entropy)"
DEFAULT_WORKLOAD = "base72b_helper"
DEFAULT_EXTRA = ("base7b_helper", "base7b", "helper4k")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ---------------------------------------------------------------- GPU passes

def marker():
    import torch
    torch.cuda._sleep(1)


def timed_pass(dec, steps, dom=None):
    """Runs the steps between two synchronisations; returns (ms, dominant
    call's event pairs)."""
    import torch
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    timers = {} if dom else None
    start.record()
    for i in steps:
        dec.step(i, timers=timers, only=dom)
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end), (timers or {}).get(dom, [])


def per_call(wl, dec, steps):
    """Replay of `steps` with event pairs around every call; eviction bytes
    at the kept rows that changed slot (read back after each eviction)."""
    import torch
    timers, moved = {}, []
    for i in steps:
        dec.step(i, timers=timers, evict_log=moved)
    torch.cuda.synchronize()
    moved_rows = None
    if moved:
        b = wl.base
        moved_rows = sum(moved) / len(moved) / (b.S * b.L * b.Hkv)
    calls = {}
    for k, ev in timers.items():
        dur = [s.elapsed_time(e) for s, e in ev]
        n = len(dur)
        call_steps = [i for i in steps if k in step_bytes(wl, dec, i)]
        b_per = sum(step_bytes(wl, dec, i, moved_rows)[k] for i in call_steps) / n
        avg_ms = sum(dur) / n
        calls[k] = dict(launches=n, avg_us=round(avg_ms * 1e3, 2), bytes_per_call=int(b_per),
                        GBps=round(b_per / (avg_ms * 1e-3) / 1e9, 1),
                        frac=round(b_per / (avg_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4))
        if k == "evict":
            ub = sum(step_bytes(wl, dec, i)[k] for i in call_steps) / n
            calls[k].update(moved_rows_per_head=round(moved_rows, 2), bytes_upper_bound=int(ub),
                            frac_upper_bound=round(ub / (avg_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4))
    return calls, moved_rows


def entropy_marginal(wl, dec, steps, reps=3):
    """Entropy's marginal time in the fused attention launch (base attention,
    or the helper's context launch when there is no base model): for every
    step of `steps`, the fused call, the same attention alone and the entropy
    call alone, one after the other, each between timing events, `reps`
    times. marginal = mean(fused) - mean(alone)."""
    import torch
    fused, alone = ("base_attn_entropy", "base_attn") if wl.base else ("helper_attn_entropy", "helper_attn")
    timers = {}
    for _ in range(reps):
        for i in steps:
            t = dec.T_prompt + i
            si = dec.inputs(t)
            if wl.base:
                dec.base_attn(t, si, timers=timers, sets=dec.logit_sets(si))
                dec.base_attn(t, si, timers=timers)
            else:
                dec.helper_token(i, si, timers=timers, sets=dec.logit_sets(si))
                dec.helper_token(i, si, timers=timers)
            dec.entropy(si, timers=timers)
    torch.cuda.synchronize()
    avg = {k: sum(s.elapsed_time(e) for s, e in ev) / len(ev) * 1e3 for k, ev in timers.items()}
    eb = acc.entropy_bytes(wl)
    mus = avg[fused] - avg[alone]
    return dict(call=fused, calls_per_kind=len(timers[alone]), fused_call_us=round(avg[fused], 2),
                attn_alone_us=round(avg[alone], 2), marginal_us=round(mus, 2),
                separate_call_us=round(avg["entropy"], 2), bytes_per_step=eb,
                GBps=round(eb / (mus * 1e-6) / 1e9, 1) if mus > 0 else None,
                frac=round(eb / (mus * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4) if mus > 0 else None,
                separate_frac=round(eb / (avg["entropy"] * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4))


def summary(wl, dec, steps, ms, moved_rows):
    K = len(steps)
    tot = sum(window_bytes(wl, dec, steps, moved_rows).values())
    S = (wl.base.S if wl.base else 0) + (wl.helper.S if wl.helper else 0)
    return dict(steps=K, ms_per_step=round(ms / K, 4), steps_per_s=round(K / (ms * 1e-3), 3),
                cand_tokens_per_s=round(S * K / (ms * 1e-3), 1),
                alg_bytes_per_step=int(tot / K), hbm_GBps=round(tot / (ms * 1e-3) / 1e9, 1),
                hbm_frac=round(tot / (ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4))


def run_workload(name, K, W, instrument=True, cycle=True, dom_events=True):
    import torch

    from paper_2608_15797_amd.pipeline import Decoder
    wl0 = WORKLOADS[name]
    C = cycle_steps(wl0)
    K = K or C
    s0 = place_window(wl0, K, W)
    win = list(range(s0, s0 + K))
    run_cycle = cycle and K != C
    c0 = cycle_start(wl0, s0 + K) if run_cycle else s0
    cyc = list(range(c0, c0 + C)) if run_cycle else []
    horizon = max(s0 + K, c0 + C if run_cycle else 0) + 1
    wl = wl0.with_(steps=horizon)
    t0 = time.time()
    dec = Decoder(wl, device="cuda")
    torch.cuda.synchronize()
    log("[%s] buffers + input pool (%d draws) ready in %.1fs" % (name, len(dec.pool), time.time() - t0))
    dec.prompt()
    for i in range(s0 - W, s0):
        dec.step(i)
    torch.cuda.synchronize()
    sch = Schedule(wl, horizon)
    wstat = window_stats(wl, sch, s0, K)
    log("[%s] prompt (%d tokens) + %d warmup steps done; window %s" % (name, dec.T_prompt, W, json.dumps(wstat)))

    dom = dominant_call(wl, dec, win)
    marker()
    ms, dom_ev = timed_pass(dec, win, dom if dom_events else None)
    marker()
    log("[%s] timed %d steps: %.4f ms/step" % (name, K, ms / K))
    calls, moved_rows = {}, None
    marginal = None
    if instrument:
        calls, moved_rows = per_call(wl, dec, win)
        log("[%s] per-call: %s" % (name, json.dumps(calls)))
        marker()
        if dec.fuse_entropy:
            marginal = entropy_marginal(wl, dec, win)
            marker()
            log("[%s] entropy marginal: %s" % (name, json.dumps(marginal)))
    else:
        marker()
    res = dict(workload=name, window=wstat, **summary(wl, dec, win, ms, moved_rows), calls=calls)
    if marginal:
        res["entropy_marginal"] = marginal
    # The dominant call's kernel time, from the events inside the timed pass
    # (else from the replay's).
    if dom_ev:
        dur = [s.elapsed_time(e) for s, e in dom_ev]
        dom_steps = [i for i in win if dom in step_bytes(wl, dec, i)]
        dom_bytes = sum(step_bytes(wl, dec, i, moved_rows)[dom] for i in dom_steps) / len(dom_steps)
        dom_us = sum(dur) / len(dur) * 1e3
        res["dominant"] = dict(call=dom, launches=len(dur), avg_us=round(dom_us, 2),
                               alg_bytes_per_call=int(dom_bytes),
                               GBps=round(dom_bytes / (dom_us * 1e-6) / 1e9, 1), timed_pass=True)
    elif dom in calls:
        c = calls[dom]
        res["dominant"] = dict(call=dom, launches=c["launches"], avg_us=c["avg_us"],
                               alg_bytes_per_call=c["bytes_per_call"], GBps=c["GBps"], timed_pass=False)
    # Algorithmic bytes per dispatch of the timed pass (between its markers),
    # for profsum --alg on counter passes of this command.
    tot, cnt = {}, {}
    for i in win:
        for k, v in step_bytes(wl, dec, i, moved_rows).items():
            tot[k] = tot.get(k, 0) + v
            cnt[k] = cnt.get(k, 0) + 1
    log(json.dumps({"workload": name, "window": wstat, "dispatches": cnt,
                    "alg_bytes_per_dispatch": {k: int(round(tot[k] / cnt[k])) for k in tot}}))
    if run_cycle:
        cms, _ = timed_pass(dec, cyc)
        marker()
        ccalls, cmoved = per_call(wl, dec, cyc) if instrument else ({}, None)
        marker()
        res["cycle"] = dict(first_step=c0, **summary(wl, dec, cyc, cms, cmoved), calls=ccalls)
        log("[%s] cycle of %d steps: %.4f ms/step" % (name, C, cms / C))
    return res, dec, wl, win


# ---------------------------------------------------------------- references

def copy_bandwidth(nbytes=1 << 30):
    """Read+write bandwidth of a plain device-to-device copy of nbytes (a
    measured reference beside the 8 TB/s nameplate)."""
    import torch
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
    import torch
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda").fill_(1.0)
    dst = torch.empty(nbytes // 2, dtype=torch.float16, device="cuda")
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst
    torch.cuda.empty_cache()


def sampler_marginal(dec, steps, reps=3):
    """The sampler's marginal time in the decode step: for every step of
    `steps`, the base-attention launch with the step's entropy rows and the
    same launch drawing every row's next token too (temperature 0.8, top-k 20,
    top-p 0.95), one after the other between timing events, `reps` times."""
    import torch

    from paper_2608_15797_amd import kvr
    smp = kvr.Sampler(seed=2608)
    timers = {}
    for _ in range(reps):
        for i in steps:
            t = dec.T_prompt + i
            si = dec.inputs(t)
            sets = dec.logit_sets(si)
            toks = [torch.empty(x.shape[0], dtype=torch.int32, device="cuda") for x in si.logits]
            dec.base_attn(t, si, timers=timers, sets=sets)
            dec.base_attn(t, si, timers=timers, sets=sets, sampler=smp, tokens=toks)
    torch.cuda.synchronize()
    avg = {k: sum(s.elapsed_time(e) for s, e in ev) / len(ev) * 1e3 for k, ev in timers.items()}
    return dict(calls_per_kind=len(timers["base_attn_entropy"]),
                entropy_call_us=round(avg["base_attn_entropy"], 2),
                entropy_sample_call_us=round(avg["base_attn_entropy_sample"], 2),
                marginal_us=round(avg["base_attn_entropy_sample"] - avg["base_attn_entropy"], 2))


def sampler_cost(dec, wl, reps=50):
    """Per-call time of the entropy pass alone and with the fused sampler
    (temperature 0.8, top-k 20, top-p 0.95) on the workload's logit sets."""
    import torch

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


def traffic_record(name, call, window=None):
    """The traffic record of `call` (profiles/traffic_<workload>.json, written
    by profsum --traffic from rocprofv3 PMC counters), or None when it is
    missing, was taken on other kernel sources or, when `window` is given,
    over other decode steps."""
    from paper_2608_15797_amd.profsum import source_hash
    path = os.path.join(ROOT, "profiles", "traffic_%s.json" % name)
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    rec = t.get("calls", {}).get(call)
    if rec is None or rec.get("source_hash") != source_hash(call):
        return None
    if window is not None and t.get("window") != window:
        return None
    return rec


def attach_traffic(name, calls, window=None):
    """Add the measured HBM bytes per call to every call that has a current
    traffic record of the same decode steps, with the algorithmic bytes of the
    same dispatches and their ratio."""
    for call, c in calls.items():
        rec = traffic_record(name, call, window)
        if rec is not None:
            c["measured_bytes_per_call"] = int(rec["bytes_per_call"])
            if "alg_bytes_per_dispatch" in rec:
                c["measured_alg_bytes_per_call"] = int(rec["alg_bytes_per_dispatch"])
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


def cpu_baseline(dec, wl, steps, min_s=10.0):
    """The fp64 oracle timed on this host with all its OpenMP threads and
    with one thread (a reported baseline, not a target); see oracle_sample
    for the sample. `value` is the all-threads rate."""
    import oracle
    n_all = oracle.threads()
    r = oracle_sample(dec, wl, steps, min_s)
    oracle.set_threads(1)
    try:
        r1 = oracle_sample(dec, wl, steps, min_s)
    finally:
        oracle.set_threads(n_all)
    return dict(value=round(r["steps"] / r["secs"], 6), unit="steps/s", cores=n_all, kind="oracle",
                single_thread_value=round(r1["steps"] / r1["secs"], 6), nproc=os.cpu_count(),
                cpu_model=cpu_model(),
                sample="%d problem-steps of the timed window's steps (%d problems per step, the window's "
                       "eviction step first, %d of them evicting: TopB and compaction of every head of the "
                       "problem's candidates), %s; %.1f s of oracle time on %d threads; %d problem-steps, "
                       "%.1f s on one thread; steps/s = problem-steps / problems / seconds"
                       % (r["done"], r["problems"], r["evicting"], "; ".join(r["desc"]), r["secs"], n_all,
                          r1["done"], r1["secs"]))


def oracle_sample(dec, wl, steps, min_s):
    """The oracle's share of the timed window, one problem at a time: its
    candidates' base attention (and, at an eviction step, TopB selection and
    compaction of each of their heads, scored by that step's attention mass),
    helper attention and logit rows, over the window's steps starting at its
    eviction step, until at least `min_s` seconds of oracle time. Host
    copies are made outside the timing."""
    import numpy as np
    import torch

    import oracle

    def host(t):
        t = t.detach().cpu().contiguous()
        return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy()

    b, h = wl.base, wl.helper
    problems = 8 if wl.name == "base72b_helper" else (16 if (b and b.S >= 16) else 1)
    ev = [i for i in steps if b and dec.blen_host[dec.T_prompt + i] > b.B + b.buffer]
    order = steps if not ev else steps[steps.index(ev[0]):] + steps[:steps.index(ev[0])]
    secs, done, evicting = 0.0, 0, 0
    desc = []
    while secs < min_s:
        for i in order:
            t = dec.T_prompt + i
            si = dec.inputs(t)
            for p in range(problems):
                if b:
                    nb = b.S // problems
                    sl = slice(p * nb, (p + 1) * nb)
                    n = dec.blen_host[t]
                    K, V, q = host(dec.bcache.k[sl]), host(dec.bcache.v[sl]), host(si.bq[sl])
                    pos = host(dec.bcache.pos[sl]).copy()
                    K, V = K.copy(), V.copy()
                    t0 = time.perf_counter()
                    _, psum = oracle.decode_attn(K, V, n, q, dec.bscale)
                    if n > b.B + b.buffer:
                        for s in range(nb):
                            for l in range(b.L):
                                for hh in range(b.Hkv):
                                    kept = oracle.select_topb(psum[s, l, hh], n, b.B, b.W)
                                    oracle.compact_head(K[s, l, hh], V[s, l, hh], pos[s, l, hh], kept)
                    secs += time.perf_counter() - t0
                    evicting += n > b.B + b.buffer
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
    return dict(steps=done / problems, secs=secs, desc=desc, done=done, problems=problems,
                evicting=evicting)


def rounded(d):
    return {k: (round(v, 4) if isinstance(v, float) else v) for k, v in d.items()}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20, help="timed steps (0: one whole cycle)")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=sorted(WORKLOADS))
    ap.add_argument("--extra", default=",".join(DEFAULT_EXTRA),
                    help="comma-separated workloads also reported, each over one whole cycle (empty: none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-instrument", action="store_true")
    ap.add_argument("--no-cycle", action="store_true", help="skip the whole-cycle pass of the headline")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a 1 GiB copy kernel three times (the known-size reference "
                         "that scales rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    if args.steps < 0 or args.warmup < 0:
        print("--steps and --warmup must be non-negative", file=sys.stderr)
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_calibration:
        calibration_copy()
    copy_ref = copy_bandwidth()

    res, dec, wl, win = run_workload(args.workload, args.steps, args.warmup, not args.no_instrument,
                                     not args.no_cycle)
    steps = res["window"]["steps"]
    calls = res["calls"]
    attach_traffic(args.workload, calls, res["window"])
    dom = res["dominant"]
    rec = traffic_record(args.workload, dom["call"], res["window"])
    frac = dom["GBps"] / PEAK_HBM_GBPS
    roof = dict(bound="hbm", achieved=dom["GBps"], peak=PEAK_HBM_GBPS, unit="GB/s", frac=round(frac, 4),
                traffic=None if rec is None else int(rec["bytes_per_call"]), call=dom["call"],
                alg_bytes_per_call=dom["alg_bytes_per_call"], avg_us=dom["avg_us"], launches=dom["launches"])
    if rec is not None and "alg_bytes_per_dispatch" in rec:
        roof["traffic_alg_bytes_per_call"] = int(rec["alg_bytes_per_dispatch"])
    sampler = sampler_cost(dec, wl) if not args.no_instrument else None
    if sampler is not None and dec.fuse_entropy and wl.base:
        sampler["in_decode_launch"] = sampler_marginal(dec, win)
    if sampler:
        log("[%s] sampler: %s" % (args.workload, json.dumps(sampler)))
    cpu = None
    if not args.no_cpu_baseline:
        t0 = time.time()
        cpu = cpu_baseline(dec, wl, win)
        log("[cpu baseline] %.1fs: %s" % (time.time() - t0, json.dumps(cpu)))
    del dec
    torch.cuda.empty_cache()

    extra = {}
    for name in [x for x in args.extra.split(",") if x and x != args.workload]:
        r, d, _, _ = run_workload(name, 0, args.warmup, not args.no_instrument, False, dom_events=False)
        attach_traffic(name, r["calls"], r["window"])
        del d
        torch.cuda.empty_cache()
        extra[name] = rounded(r)

    cfg = describe(WORKLOADS[args.workload])
    cfg.update(window=res["window"], cand_tokens_per_s=res["cand_tokens_per_s"],
               alg_bytes_per_step=res["alg_bytes_per_step"], hbm_GBps=res["hbm_GBps"],
               hbm_frac_of_peak=res["hbm_frac"], calls=calls)
    line = {
        "metric": METRIC, "value": res["steps_per_s"], "unit": "steps/s",
        "n_gpus": 1, "steps": steps, "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded, Qwen2.5-Math shapes)",
        "config": cfg, "roofline": roof, "cpu_baseline": cpu,
        "entropy_marginal": res.get("entropy_marginal"),
        "cycle": res.get("cycle"), "workloads": extra, "sampler": sampler,
        "copy_ref_GBps": copy_ref,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
