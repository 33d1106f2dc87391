"""Measurement probes behind the ceilings quoted for the decode kernels
(measurement only; the decode path never uses them).

    python -m paper_2608_15797_amd.probes stream attn UNITS CAP N [N ...]
    python -m paper_2608_15797_amd.probes stream evict HEADS CAP B W N
    python -m paper_2608_15797_amd.probes stream read MB [MB ...]
    python -m paper_2608_15797_amd.probes stream readpol MB [MB ...]
    python -m paper_2608_15797_amd.probes stream lanes
    python -m paper_2608_15797_amd.probes entropy [--rows 0,1,8,32,64,128,256]

`stream` builds and runs streamprobe.hip (load-only attention streams,
eviction-shaped copies, plain read-only streams and the same streams under
each cache policy of the loads, and the lane layout of the cross-lane swap
instructions; see that file). `entropy` times the library's
base-attention launch with and without the step's entropy rows in it
(kvr_decode_attn_entropy against kvr_decode_attn), at fixed cache lengths of
the 72B and 7B B=128 base shapes, for several numbers of 152064-logit rows:
the difference is entropy's marginal time in the fused launch.
"""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "streamprobe.hip")
BIN = os.path.join(HERE, "streamprobe")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang",
         "-packed-fp32-ops"]


def build(verbose: bool = False) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmp = BIN + ".tmp%d" % os.getpid()
    res = subprocess.run([hipcc] + FLAGS + [SRC, "-o", tmp], stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                         text=True)
    out = "\n".join(l for l in res.stdout.splitlines() if "packed-fp32-ops' is not a recognized feature" not in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed on streamprobe.hip:\n" + out)
    if verbose and out.strip():
        print(out)
    os.replace(tmp, BIN)
    return BIN
