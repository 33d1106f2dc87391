"""Mistakes planted in the oracle are caught by its pins (CPU only).

Each mutant is a copy of the oracle package with one plausible mistake
planted in its source: a wrong grouped-query head mapping, a dropped softmax
scale, a key too few, the wrong tie-break, a log of the wrong base, an
off-by-one in the detector's guard, ... The copy is built and the pin suites
run against it; every mutant must make at least one pin fail. A pin set that
passed a mutant would also pass an oracle carrying that mistake, so this
checks the pins, not the oracle.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle")
PINS = ["tests/test_oracle_pins.py", "tests/test_oracle_golden.py", "tests/test_oracle_movement.py",
        "tests/test_oracle_sampler.py", "tests/test_oracle_rkv.py"]

C = "kvr_oracle.c"
MUTANTS = [
    # Attention (Eq. (1), third line) and its grouped-query layout.
    ("gqa_strided_heads", C,
     "            int qh = h * G + g;\n            size_t qoff = (((size_t)s * L + l) * Hq + qh) * (size_t)D;",
     "            int qh = g * Hkv + h;\n            size_t qoff = (((size_t)s * L + l) * Hq + qh) * (size_t)D;"),
    ("scale_dropped", C, "x[j] = scale * dot;", "x[j] = dot;"),
    ("last_key_dropped", C, "K, V, coff, ns, o, prow);", "K, V, coff, ns - 1, o, prow);"),
    ("prefix_dropped", C, "n1 = plen;", "n1 = 0;"),
    ("prefix_interleaved", C, "int p = s / (S / P);", "int p = s % P;"),
    ("bf16_widening", C, "[i] << 16;", "[i] << 15;"),
    # Importance score (Sec. 2.1): the window's attention mass.
    ("psum_not_summed_over_group", C, "ps[j] += prow[j];", "ps[j] = prow[j];"),
    ("window_rows_not_causal", C, "int nr = n[s] - (nq - 1 - r);", "int nr = n[s];"),
    ("window_off_by_one", C, "int nr = n[s] - (nq - 1 - r);", "int nr = n[s] - (nq - r);"),
    ("window_heads_strided", C,
     "                int qh = h * G + g;\n                size_t qoff = ((((size_t)s",
     "                int qh = g * Hkv + h;\n                size_t qoff = ((((size_t)s"),
    # TopB and compaction (Eq. (1), first two lines).
    ("topb_ties_to_higher_slot", C, "score[j] > score[best]", "score[j] >= score[best]"),
    ("topb_smallest_scores", C, "score[j] > score[best]", "score[j] < score[best]"),
    ("topb_window_not_protected", C, "int ncand = n - W, take = B - W;", "int ncand = n - W + 1, take = B - W;"),
    ("kept_descending", C, "for (int j = 0; j < ncand; j++) if (taken[j]) kept[cnt++] = j;",
     "for (int j = ncand - 1; j >= 0; j--) if (taken[j]) kept[cnt++] = j;"),
    ("compact_pos_dropped", C, "if (pos) pos[i] = pos[src];", "(void)pos;"),
    ("compact_skips_moved_row", C, "if (src == i) continue;", "if (src <= i + 1) continue;"),
    # Entropy (Eq. (4)).
    ("entropy_log2", C, "h -= p * log(p);", "h -= p * log2(p);"),
    ("entropy_temperature_not_in_z", C, "Z += exp(inv_temp * elem(logits, dtype, base + v) - m);",
     "Z += exp(elem(logits, dtype, base + v) - m);"),
    ("entropy_reads_row_padding", C, "for (int v = 0; v < V; v++) Z +=", "for (int v = 0; v < ld; v++) Z +="),
    # Detector (Eq. (4) moving average; guard 24, window 12, tau 7).
    ("detector_guard_off_by_one", C, "if (cnt[r] >= guard) {", "if (cnt[r] > guard) {"),
    ("detector_mean_over_full_window", C, "int k = cnt[r] < window ? cnt[r] : window;", "int k = window;"),
    ("detector_not_sticky", C, "if (sum / k > tau) flag[r] = 1;", "flag[r] = sum / k > tau;"),
    # The per-token loop of the evicted base model.
    ("run_window_starts_late", "run.py", "if self.n >= window_start(self.B, self.W, self.buffer):",
     "if self.n > window_start(self.B, self.W, self.buffer):"),
    ("run_score_is_last_row", "run.py", "score = np.sum(self.rows, axis=0)", "score = self.rows[-1]"),
    ("run_keeps_one_more", "run.py", "self.n = self.B\n", "self.n = self.B + 1\n"),
    # Fork / commit data movement.
    ("fork_copies_one_slot_short", "movement.py", "for j in range(n):", "for j in range(n - 1):"),
    ("commit_window_all_queries", "movement.py", "nq = min(W, T)", "nq = T"),
    # Sampler (Sec. 4.1 decoding setup).
    ("sampler_ties_to_higher_id", "sampler.py", "np.lexsort((np.arange(V), -x))", "np.lexsort((-np.arange(V), -x))"),
    ("sampler_temperature_multiplies", "sampler.py", "z = x[order] / temperature", "z = x[order] * temperature"),
    ("sampler_nucleus_one_short", "sampler.py", "keep = int(np.argmax(cum >= top_p)) + 1",
     "keep = max(1, int(np.argmax(cum >= top_p)))"),
    ("sampler_draw_not_strict", "sampler.py", "cum[:keep] > target)) if np.any(cum[:keep] > target)",
     "cum[:keep] >= target)) if np.any(cum[:keep] >= target)"),
    ("philox_keys_swapped", "sampler.py", "((p1 >> 64) ^ c[1] ^ k[0]) & _M64, p1 & _M64,\n             ((p0 >> 64) ^ c[3] ^ k[1])",
     "((p1 >> 64) ^ c[1] ^ k[1]) & _M64, p1 & _M64,\n             ((p0 >> 64) ^ c[3] ^ k[0])"),
    # Redundancy-aware score (a documented reading; its pieces are pinned).
    ("cosine_mean_over_m", "rkv.py", "R[c] = tot / (m - 1)", "R[c] = tot / m"),
    ("pool_radius_doubled", "rkv.py", "r = pool // 2", "r = pool"),
    ("lambda_weights_swapped", "rkv.py", "return lam * Ih - (1.0 - lam) * Rh", "return (1.0 - lam) * Ih - lam * Rh"),
]


def _run_mutant(tmp, name, fname, old, new):
    """Pin-suite result on one mutant: (exit status, output tail)."""
    pkg = os.path.join(tmp, "oracle")
    shutil.copytree(ORACLE, pkg, ignore=shutil.ignore_patterns("*.so", "*.so.tmp*", "__pycache__"))
    path = os.path.join(pkg, fname)
    with open(path) as f:
        src = f.read()
    if src.count(old) != 1:
        return -100, "mutation site not found exactly once in %s" % fname
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    # The mutant package is imported (and its C part built) before pytest
    # starts, so the pins' `import oracle` finds it whatever sys.path the
    # test session sets up afterwards.
    code = ("import sys; sys.path.insert(0, %r); import oracle; assert oracle.__file__.startswith(%r); "
            "oracle.build(force=True); import oracle.run, oracle.movement, oracle.sampler, oracle.rkv; "
            "import pytest; sys.exit(pytest.main(['-q', '-x', '-p', 'no:cacheprovider', %s]))"
            % (tmp, pkg, ", ".join(repr(p) for p in PINS)))
    env = dict(os.environ, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=600)
    return r.returncode, (r.stdout + r.stderr)[-1500:]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_pins_catch_every_planted_mistake(tmp_path):
    """Every mutant must end its pin session with pytest status 1 (tests ran
    and at least one failed); 0 would mean every pin passed the mistake, any
    other status a broken run."""
    from concurrent.futures import ThreadPoolExecutor
    jobs = {}
    with ThreadPoolExecutor(max_workers=min(6, os.cpu_count() or 1)) as ex:
        for name, fname, old, new in MUTANTS:
            d = tmp_path / name
            d.mkdir()
            jobs[name] = ex.submit(_run_mutant, str(d), name, fname, old, new)
    bad = []
    for name, fut in jobs.items():
        rc, tail = fut.result()
        if rc != 1 or " failed" not in tail:
            bad.append("%s (exit %d):\n%s" % (name, rc, tail))
    assert not bad, "mutants not caught by the pins:\n" + "\n\n".join(bad)
