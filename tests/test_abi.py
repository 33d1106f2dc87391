"""The C-ABI library loads on the host, exports every function include/kvr.h
declares, and rejects bad arguments on the host before touching the GPU."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "kvr.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(kvr_[a-z_]+)\s*\(", src)))


def test_header_declares_the_four_entry_points():
    names = declared_functions()
    for f in ("kvr_decode_attn", "kvr_accumulate_scores", "kvr_evict_topb", "kvr_logit_entropy"):
        assert f in names


def test_library_exports_every_declared_symbol():
    from paper_2608_15797_amd import kvr
    for name in declared_functions():
        assert hasattr(kvr.lib, name), name
    assert set(declared_functions()) == set(kvr.EXPORTS)


C_CALLER = r"""
#include <stdio.h>
#include <string.h>
#include "kvr.h"
int main(void) {
  kvr_cache c;
  memset(&c, 0, sizeof c);
  int st = kvr_evict_topb(&c, NULL, NULL, NULL, NULL, NULL, NULL);
  printf("%s|%d|%s\n", kvr_strerror(KVR_OK), st, kvr_last_error());
  return st == KVR_EINVAL ? 0 : 1;
}
"""


@pytest.mark.skipif(not os.path.exists("/opt/rocm/include/hip/hip_runtime_api.h"), reason="HIP headers absent")
def test_header_is_a_c_abi(tmp_path):
    """include/kvr.h compiles as C11 without warnings, and a C program links
    against libkvr.so and gets a host-side rejection with its message."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    from paper_2608_15797_amd import kvr
    src = tmp_path / "caller.c"
    src.write_text(C_CALLER)
    exe = str(tmp_path / "caller")
    libdir = os.path.dirname(kvr.LIB_PATH)
    r = subprocess.run(["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
                        "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include", str(src),
                        "-L", libdir, "-lkvr", "-Wl,-rpath," + libdir, "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    out = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert out.returncode == 0, out.stdout + out.stderr
    ok, status, msg = out.stdout.strip().split("|")
    assert ok == "ok" and int(status) == -1 and "NULL" in msg


def test_status_strings():
    from paper_2608_15797_amd import kvr
    assert kvr.lib.kvr_strerror(0) == b"ok"
    assert kvr.lib.kvr_strerror(-1) == b"invalid argument"
    assert kvr.lib.kvr_strerror(-4) == b"workspace missing or too small"


def _cache(kvr, **kw):
    d = dict(k=16, v=16, pos=None, S=2, L=1, Hkv=2, cap=33, D=128, dtype=1)
    d.update(kw)
    return kvr.c_cache(d["k"], d["v"], d["pos"], d["S"], d["L"], d["Hkv"], d["cap"], d["D"], d["dtype"])


@pytest.mark.parametrize("kw,Hq,status,msg", [
    (dict(k=None), 8, -1, "NULL"),
    (dict(D=96), 8, -2, "head_dim"),
    (dict(dtype=7), 8, -2, "dtype"),
    (dict(S=0), 8, -1, "positive"),
    ({}, 7, -1, "multiple"),
    ({}, 34, -2, "exceeds 16"),
    (dict(k=24), 8, -1, "aligned"),
])
def test_decode_attn_rejects_bad_arguments_on_host(kw, Hq, status, msg):
    from paper_2608_15797_amd import kvr
    c = _cache(kvr, **kw)
    rc = kvr.lib.kvr_decode_attn(ctypes.byref(c), None, 16, 16, Hq, 1.0, None, None, None, 16,
                                 None, None, None, 0, None)
    assert rc == status
    assert msg in kvr.lib.kvr_last_error().decode()


def test_policy_validation_on_host():
    from paper_2608_15797_amd import kvr
    c = _cache(kvr, cap=20)
    for pol, msg in ((kvr.c_policy(16, 8, 16), "cap="), (kvr.c_policy(16, 0, 4), "0 < W < B"),
                     (kvr.c_policy(8, 4, 2), "buffer >= W-1")):
        rc = kvr.lib.kvr_evict_topb(ctypes.byref(c), 16, None, 16, ctypes.byref(pol), None, None)
        assert rc == -1 and msg in kvr.lib.kvr_last_error().decode()
    # len_out must not overlap len ([S] int32 each; S = 2 here).
    c = _cache(kvr, cap=40)
    pol = kvr.c_policy(16, 8, 16)
    for lo in (16, 12, 20):
        rc = kvr.lib.kvr_evict_topb(ctypes.byref(c), 16, lo, 16, ctypes.byref(pol), None, None)
        assert rc == -1 and "overlaps" in kvr.lib.kvr_last_error().decode()


def test_entropy_rejects_bad_arguments_on_host():
    from paper_2608_15797_amd import kvr
    assert kvr.lib.kvr_logit_entropy(16, 1, 4, 10, 5, 1.0, 16, None, None, 0, None) == -1
    assert kvr.lib.kvr_logit_entropy(16, 3, 4, 10, 10, 1.0, 16, None, None, 0, None) == -2
    # A split reduction needs a workspace.
    need = kvr.lib.kvr_logit_entropy_workspace_size(8, 151936)
    assert need > 0
    assert kvr.lib.kvr_logit_entropy(16, 1, 8, 151936, 151936, 1.0, 16, None, None, 0, None) == -4
    # The softmax temperature's inverse must be positive and finite.
    for bad in (0.0, -1.0, float("inf"), float("nan")):
        assert kvr.lib.kvr_logit_entropy(16, 1, 4, 10, 10, bad, 16, None, None, 0, None) == -1
        assert "inv_temp" in kvr.lib.kvr_last_error().decode()


def test_entropy_batch_rejects_bad_arguments_on_host():
    from paper_2608_15797_amd import kvr

    def sets(*specs):
        arr = (kvr.c_logit_set * len(specs))()
        for k, (dtype, R, V, ld, it) in enumerate(specs):
            arr[k] = kvr.c_logit_set(16, dtype, R, V, ld, it, 16 + 4096 * k, None)
        return arr

    f, ws = kvr.lib.kvr_logit_entropy_batch, kvr.lib.kvr_logit_entropy_batch_workspace_size
    # 256 long rows (both 128-row vocabularies of the default step): one
    # whole-row workgroup per row, no split partials, no workspace.
    assert ws(sets((1, 128, 152064, 152064, 1.0), (1, 128, 151936, 151936, 1.0)), 2) == 0
    # 2 x 64 rows share one split plan: 128 rows x 8 splits of 16-byte partials.
    two = sets((1, 64, 152064, 152064, 1.0), (1, 64, 151936, 151936, 1.0))
    assert ws(two, 2) == 128 * 8 * 16
    assert f(two, 2, None, 0, None) == -4
    assert f(two, 2, 16, 128 * 8 * 16 - 1, None) == -4
    assert f(None, 2, None, 0, None) == -1
    for n in (0, 5):
        assert f(two, n, None, 0, None) == -1 and "nsets" in kvr.lib.kvr_last_error().decode()
    # The size query reads shapes only.
    assert kvr.logit_entropy_batch_workspace_size([(128, 152064), (128, 151936)]) == 0
    assert kvr.logit_entropy_batch_workspace_size([(64, 152064), (64, 151936)]) == 128 * 8 * 16
    assert kvr.logit_entropy_workspace_size(300, 152064) == 0  # whole-row workgroups
    assert kvr.logit_entropy_workspace_size(128, 152064) == 128 * 8 * 16
    assert kvr.logit_entropy_batch_workspace_size([(3, 10)]) == 0
    mixed = sets((1, 4, 10, 10, 1.0), (0, 4, 10, 10, 1.0))
    assert f(mixed, 2, None, 0, None) == -1 and "dtype" in kvr.lib.kvr_last_error().decode()
    assert ws(mixed, 2) == 0
    many = sets((1, 40000, 10, 10, 1.0), (1, 30000, 10, 10, 1.0))
    assert f(many, 2, None, 0, None) == -1 and "rows" in kvr.lib.kvr_last_error().decode()
    # Each set is checked as kvr_logit_entropy checks its arguments.
    assert f(sets((1, 4, 10, 10, 1.0), (1, 4, 10, 5, 1.0)), 2, None, 0, None) == -1
    assert f(sets((1, 4, 10, 10, 1.0), (1, 4, 10, 10, float("nan"))), 2, None, 0, None) == -1
    assert f(sets((3, 4, 10, 10, 1.0)), 1, None, 0, None) == -2


def test_prefix_workspace_size_matches_split_plan():
    from paper_2608_15797_amd import kvr
    c = _cache(kvr, S=128, L=28, Hkv=2, cap=512)
    p = kvr.c_prefix(16, 16, 16, 8192)
    n = kvr.lib.kvr_decode_attn_workspace_size(ctypes.byref(c), ctypes.byref(p), 12)
    # One record per query row and split: (max, sum, -, -) float32 + 128 float16.
    rec = 128 * 28 * 12 * (16 + 128 * 2)
    assert n % rec == 0 and n // rec >= 2


def test_fork_rejects_bad_arguments_on_host():
    from paper_2608_15797_amd import kvr
    src = _cache(kvr)
    cases = [
        (_cache(kvr, k=48, v=64, L=2), 16, 16, None, None, "differ"),
        (_cache(kvr, k=48, v=64, dtype=0), 16, 16, None, None, "differ"),
        (_cache(kvr, k=48, v=64), None, 16, None, None, "required"),
        (_cache(kvr, k=48, v=64), 16, 16, 16, None, "both"),
        (_cache(kvr, k=48, v=64, pos=80), 16, 16, None, None, "positions"),
        (_cache(kvr, k=16, v=64), 16, 16, None, None, "same cache"),
        (_cache(kvr, k=48, v=16), 16, 16, None, None, "share v"),
    ]
    for dst, idx, ln, ssc, dsc, msg in cases:
        rc = kvr.lib.kvr_fork(ctypes.byref(src), ctypes.byref(dst), idx, ln, ssc, dsc, None)
        assert rc == -1, msg
        assert msg in kvr.lib.kvr_last_error().decode()


def test_append_rejects_bad_arguments_on_host():
    from paper_2608_15797_amd import kvr
    c = _cache(kvr)
    assert kvr.lib.kvr_append(ctypes.byref(c), 16, -1, 16, 16, None, None) == -1
    assert kvr.lib.kvr_append(ctypes.byref(c), 16, 3, 16, 16, 16, None) == -1   # no cache pos
    assert "pos" in kvr.lib.kvr_last_error().decode()
    assert kvr.lib.kvr_append(ctypes.byref(c), 16, 3, None, 16, None, None) == -1
    assert kvr.lib.kvr_append(ctypes.byref(c), 16, 3, 24, 16, None, None) == -1  # alignment
    assert kvr.lib.kvr_append(ctypes.byref(c), 16, 1 << 30, 16, 16, None, None) == -2
    # T == 0 enqueues nothing and needs no token arrays
    assert kvr.lib.kvr_append(ctypes.byref(c), 16, 0, None, None, None, None) == 0


def test_sampler_rejects_bad_arguments_on_host():
    from paper_2608_15797_amd import kvr
    f = kvr.lib.kvr_logit_entropy_sample
    need = kvr.lib.kvr_logit_entropy_sample_workspace_size(8, 151936, 20)
    assert need > 0 and need % 16 == 0
    assert kvr.lib.kvr_logit_entropy_sample_workspace_size(8, 151936, 65) == 0
    good = kvr.c_sampler(0.8, 20, 0.95, 1, 2)
    for smp, msg in ((kvr.c_sampler(0.0, 20, 0.95, 0, 0), "temperature"),
                     (kvr.c_sampler(0.8, 0, 0.95, 0, 0), "top_k"),
                     (kvr.c_sampler(0.8, 65, 0.95, 0, 0), "top_k"),
                     (kvr.c_sampler(0.8, 20, 0.0, 0, 0), "top_p"),
                     (kvr.c_sampler(0.8, 20, 1.01, 0, 0), "top_p")):
        rc = f(16, 1, 8, 1024, 1024, 1.0, 16, None, ctypes.byref(smp), 16, 16, 1 << 20, None)
        assert rc == -1 and msg in kvr.lib.kvr_last_error().decode()
    # tokens are required; a workspace is always required
    assert f(16, 1, 8, 1024, 1024, 1.0, 16, None, ctypes.byref(good), None, 16, 1 << 20, None) == -1
    assert f(16, 1, 8, 1024, 1024, 1.0, 16, None, ctypes.byref(good), 16, None, 0, None) == -4


def test_lds_limits_rejected_on_host():
    """One step past each kernel's LDS bound is refused before any launch."""
    from paper_2608_15797_amd import kvr
    # Scored decode at G = 16: cap 961 rounds to 1024 slots of logits per head.
    c = _cache(kvr, Hkv=1, cap=961)
    pol = kvr.c_policy(704, 64, 256)
    rc = kvr.lib.kvr_decode_attn(ctypes.byref(c), None, 16, 16, 16, 1.0, None, None, None, 16,
                                 ctypes.byref(pol), 16, None, 0, None)
    assert rc == -2 and "LDS" in kvr.lib.kvr_last_error().decode()
    # Eviction: (cap + B) words of LDS, at most 16384.
    c = _cache(kvr, cap=16129)
    pol = kvr.c_policy(256, 32, 15872)
    assert kvr.lib.kvr_evict_topb(ctypes.byref(c), 16, None, 16, ctypes.byref(pol), None, None) == -2
    # Window recompute (bf16): one 64-bit fixed-point accumulator per slot.
    c = _cache(kvr, cap=8193)
    assert kvr.lib.kvr_accumulate_scores(ctypes.byref(c), 16, 16, 8, 8, 1.0, 16, 0, None) == -2
    c = _cache(kvr, cap=8192, k=0, v=0)  # within the limit: fails later, on the NULL cache pointers
    assert kvr.lib.kvr_accumulate_scores(ctypes.byref(c), 16, 16, 8, 8, 1.0, 16, 0, None) == -1


def test_entropy_noalloc_rejects_on_host():
    """The allocation-free entropy call validates like the workspace call and
    refuses, before any GPU work, a split plan larger than its scratch."""
    from paper_2608_15797_amd import kvr
    f = kvr.lib.kvr_logit_entropy_batch_noalloc
    arr = (kvr.c_logit_set * 1)()
    # 200 rows of 2^24 logits: 820 splits of 16-byte partials per row, 2.6 MB.
    arr[0] = kvr.c_logit_set(16, 1, 200, 1 << 24, 1 << 24, 1.0, 16, None)
    assert kvr.lib.kvr_logit_entropy_batch_workspace_size(arr, 1) > kvr.ENTROPY_SCRATCH_BYTES
    assert f(arr, 1, None) == -2 and "scratch" in kvr.lib.kvr_last_error().decode()
    assert f(None, 1, None) == -1
    arr[0] = kvr.c_logit_set(16, 1, 4, 10, 5, 1.0, 16, None)
    assert f(arr, 1, None) == -1


def test_decode_attn_entropy_rejects_on_host():
    """The fused attention + entropy call checks the attention arguments and
    every logit set, and refuses rows that do not start 16-byte aligned."""
    from paper_2608_15797_amd import kvr
    f = kvr.lib.kvr_decode_attn_entropy
    c = _cache(kvr)
    arr = (kvr.c_logit_set * 1)()
    arr[0] = kvr.c_logit_set(16, 1, 4, 1001, 1001, 1.0, 16, None)  # ld * 2 = 2002 bytes
    assert f(ctypes.byref(c), None, 16, 16, 8, 1.0, None, None, None, 16, None, None, None, 0, arr, 1, None) == -1
    assert "aligned" in kvr.lib.kvr_last_error().decode()
    arr[0] = kvr.c_logit_set(16, 1, 4, 10, 5, 1.0, 16, None)  # ld < V
    assert f(ctypes.byref(c), None, 16, 16, 8, 1.0, None, None, None, 16, None, None, None, 0, arr, 1, None) == -1
    bad = _cache(kvr, D=96)
    arr[0] = kvr.c_logit_set(16, 1, 4, 1024, 1024, 1.0, 16, None)
    assert f(ctypes.byref(bad), None, 16, 16, 8, 1.0, None, None, None, 16, None, None, None, 0, arr, 1, None) == -2
    assert f(ctypes.byref(c), None, 16, 16, 8, 1.0, None, None, None, 16, None, None, None, 0, None, 1, None) == -1


def test_fork_rejects_shapes_beyond_its_grid_on_host():
    """A fork launch covers at most 32767 (layer, KV head) units and 524280
    destinations; larger shapes are refused before anything is enqueued."""
    from paper_2608_15797_amd import kvr
    f = kvr.lib.kvr_fork
    for kw, msg in ((dict(L=16384, Hkv=2), "L*Hkv=32768"), (dict(S=524281), "S=524281")):
        src = _cache(kvr, **{k: v for k, v in kw.items() if k != "S"})
        dst = _cache(kvr, k=32, v=48, **kw)
        assert f(ctypes.byref(src), ctypes.byref(dst), 16, 16, None, None, None) == -2
        assert msg in kvr.lib.kvr_last_error().decode()
    for kw in (dict(L=16383, Hkv=2), dict(S=524280, Hkv=1)):  # at the limits: on to the next check
        src = _cache(kvr, **{k: v for k, v in kw.items() if k != "S"})
        dst = _cache(kvr, k=32, v=48, **kw)
        assert f(ctypes.byref(src), ctypes.byref(dst), None, 16, None, None, None) == -1
        assert "src_index" in kvr.lib.kvr_last_error().decode()


def test_decode_attn_entropy_with_prefix_rejects_on_host():
    """With a prefix the fused call needs kvr_decode_attn's workspace, and
    scoring stays unavailable, as for kvr_decode_attn."""
    from paper_2608_15797_amd import kvr
    f = kvr.lib.kvr_decode_attn_entropy
    c = _cache(kvr, S=16, Hkv=2, cap=512)
    p = kvr.c_prefix(16, 16, 2, 8192)
    arr = (kvr.c_logit_set * 1)()
    arr[0] = kvr.c_logit_set(16, 1, 8, 151936, 151936, 1.0, 16, None)
    need = kvr.lib.kvr_decode_attn_workspace_size(ctypes.byref(c), ctypes.byref(p), 12)
    assert need > 0

    def call(ws, nbytes, pol=None, scores=None):
        return f(ctypes.byref(c), ctypes.byref(p), 16, 16, 12, 1.0, None, None, None, 16,
                 ctypes.byref(pol) if pol is not None else None, scores, ws, nbytes, arr, 1, None)

    assert call(None, 0) == -4
    assert call(16, need - 16) == -4 and "workspace" in kvr.lib.kvr_last_error().decode()
    assert call(16, need, kvr.c_policy(64, 32, 64), 16) == -1
    assert "prefix" in kvr.lib.kvr_last_error().decode()


def test_decode_attn_entropy_sample_rejects_on_host():
    """The fused attention + entropy + sampler call checks what the fused
    entropy call checks, the sampler settings and the tokens array."""
    from paper_2608_15797_amd import kvr
    f = kvr.lib.kvr_decode_attn_entropy_sample
    c = _cache(kvr)
    arr = (kvr.c_logit_set * 1)()
    arr[0] = kvr.c_logit_set(16, 1, 4, 1024, 1024, 1.0, 16, None)
    toks = (ctypes.c_void_p * 1)(16)
    none = (ctypes.c_void_p * 1)(None)

    def call(smp, t=toks):
        return f(ctypes.byref(c), None, 16, 16, 8, 1.0, None, None, None, 16, None, None, None, 0, arr, 1,
                 ctypes.byref(smp) if smp is not None else None, t, None)

    assert call(None) == -1 and "sampler" in kvr.lib.kvr_last_error().decode()
    for bad, msg in ((kvr.c_sampler(0.0, 20, 0.95, 0, 0), "temperature"), (kvr.c_sampler(0.8, 0, 0.95, 0, 0), "top_k"),
                     (kvr.c_sampler(0.8, 65, 0.95, 0, 0), "top_k"), (kvr.c_sampler(0.8, 20, 0.0, 0, 0), "top_p"),
                     (kvr.c_sampler(0.8, 20, 1.5, 0, 0), "top_p")):
        assert call(bad) == -1 and msg in kvr.lib.kvr_last_error().decode()
    good = kvr.c_sampler(0.8, 20, 0.95, 0, 0)
    assert call(good, None) == -1 and "tokens" in kvr.lib.kvr_last_error().decode()
    assert call(good, none) == -1 and "tokens" in kvr.lib.kvr_last_error().decode()
    arr[0] = kvr.c_logit_set(16, 1, 4, 1001, 1001, 1.0, 16, None)  # rows not 16-byte aligned
    assert call(good) == -1 and "aligned" in kvr.lib.kvr_last_error().decode()
