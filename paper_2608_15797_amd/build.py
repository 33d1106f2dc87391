"""Build libkvr.so (HIP, gfx950) in-tree.

    python -m paper_2608_15797_amd.build

Compiles every csrc/*.hip into one shared library next to this file. Packed
fp32 VALU instructions are disabled for all device code. csrc/attn_wide.hip
(the helper context kernels of three and four row blocks) is compiled to an
object of its own with the matrix-core accumulators in vector registers
(WIDE_FLAGS) and linked in.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libkvr.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


WIDE = os.path.join(HERE, "csrc", "attn_wide.hip")
# Matrix-core accumulators in vector registers. Measured on whole suffix
# cycles: the three-row-block context kernel (437 -> 357 registers, its
# per-chunk accumulator copies gone) takes the 7B + helper call from 754-761
# to 709-715 us; applied to the whole library it made the one-row-block
# kernel of the 72B helper 0.9-2.2% slower, so it is given to this file only.
WIDE_FLAGS = ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]


def sources():
    return sorted(f for f in glob.glob(os.path.join(HERE, "csrc", "*.hip")) if f != WIDE)


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(line for line in res.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in line)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + out)
    if verbose and out.strip():
        print(out)


def build(verbose: bool = False) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmp = LIB + ".tmp%d" % os.getpid()
    obj = LIB + ".wide%d.o" % os.getpid()
    try:
        _run([hipcc] + [f for f in HIPCC_FLAGS if f != "-shared"] + WIDE_FLAGS + ["-c", WIDE, "-o", obj], verbose)
        # The object goes before the sources: hipcc marks every input after a .hip file as HIP source.
        _run([hipcc] + HIPCC_FLAGS + [obj] + sources() + ["-o", tmp], verbose)
    finally:
        if os.path.exists(obj):
            os.remove(obj)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    print("built", LIB)
    sys.exit(0)
