"""Pins of the sampler oracle (oracle/sampler.py).

  Q1  Philox4x64-10 equals numpy's independent Philox bit generator (which
      advances its counter by one before producing each block).
  Q2  closed form: logits T * ln(w) give probabilities proportional to w;
      the token as a function of u switches exactly at the cumulative
      masses, for full, top-p-cut and top-k-cut nuclei.
  Q3  top_k = 1, or a vanishing top_p, is greedy decoding for every u,
      ties going to the lower token id.
  Q4  u = 0 draws the most probable token; u just below 1 draws the last
      token of the nucleus.
  Q5  with u from the generator over many steps, token frequencies match
      the renormalised top-k / top-p probabilities (chi-square), so the
      generator's top 24 bits are uniform enough and the nucleus is right.
  Q6  temperature only rescales: the top-k set does not depend on it and a
      lower temperature concentrates the draw.
  Q7  the inverse-CDF intervals are half-open: token i of the nucleus is
      drawn for u * mass in [cum_{i-1}, cum_i), so u exactly at a cumulative
      mass draws the next token.
"""
import math

import numpy as np
import pytest

from oracle import sampler


def _add(ctr, k):
    """Counter words as one little-endian 256-bit integer, plus k."""
    v = sum(int(w) << (64 * i) for i, w in enumerate(ctr)) + k
    return [(v >> (64 * i)) & (2 ** 64 - 1) for i in range(4)]


@pytest.mark.parametrize("ctr,key", [((5, 7, 0, 0), (123, 456)), ((0, 0, 0, 0), (0, 0)),
                                     ((2 ** 64 - 2, 3, 9, 1), (2 ** 63 + 5, 77)),
                                     ((1000, 2 ** 40, 2 ** 50, 2 ** 60), (0x4B5652, 1))])
def test_q1_philox_matches_numpy(ctr, key):
    bg = np.random.Philox(counter=np.array(ctr, np.uint64), key=np.array(key, np.uint64))
    raw = [int(x) for x in bg.random_raw(12)]
    ours = []
    for b in range(3):
        ours += sampler.philox4x64_10(_add(ctr, b + 1), key)
    assert ours == raw


def test_q2_closed_form_boundaries():
    T = 0.8
    w = np.array([1.0, 2.0, 3.0, 4.0])
    logits = T * np.log(w)
    # sorted tokens 3, 2, 1, 0 with probabilities .4 .3 .2 .1
    cases = [
        (4, 1.0, [0.4, 0.7, 0.9, 1.0], [3, 2, 1, 0]),       # full nucleus
        (4, 0.85, [0.4, 0.7, 0.9], [3, 2, 1]),              # top-p keeps 3 (mass .9)
        (4, 0.7, [0.4, 0.7], [3, 2]),                       # cumulative .7 reaches .7
        (2, 1.0, [4 / 7, 1.0], [3, 2]),                     # top-k 2, renormalised
    ]
    for k, p, cum, toks in cases:
        mass = cum[-1]
        edges = [c / mass for c in cum]
        lo = 0.0
        for e, t in zip(edges, toks):
            # just inside each interval: exactly on an edge, rounding decides
            for u in (lo + 1e-9 if lo > 0 else 0.0, (lo + e) / 2, e - 1e-9):
                if u < 1.0:
                    tok, d = sampler.sample_row(logits, 4, T, k, p, u)
                    assert tok == t, (k, p, u, tok, t)
            lo = e
        tok, d = sampler.sample_row(logits, 4, T, k, p, 0.0)
        assert d["keep"] == len(toks)
        np.testing.assert_allclose(np.cumsum(d["q"])[: len(cum)], cum, rtol=1e-12)


def test_q3_greedy_limits_and_ties():
    rng = np.random.default_rng(3)
    x = rng.standard_normal(500)
    x[[17, 230]] = x.max() + 1.0          # tie for the maximum: lower id wins
    for u in (0.0, 0.3, 0.999):
        assert sampler.sample_row(x, 500, 0.8, 1, 0.95, u)[0] == 17
        assert sampler.sample_row(x, 500, 0.8, 20, 1e-12, u)[0] == 17


def test_q4_extreme_uniforms():
    rng = np.random.default_rng(4)
    x = rng.standard_normal(1000) * 3
    tok0, d = sampler.sample_row(x, 1000, 0.8, 20, 0.95, 0.0)
    assert tok0 == d["order"][0] == int(np.argmax(x))
    tok1, d = sampler.sample_row(x, 1000, 0.8, 20, 0.95, 1.0 - 2.0 ** -24)
    assert tok1 == d["order"][d["keep"] - 1]


def test_q5_frequencies_match_nucleus():
    rng = np.random.default_rng(5)
    V = 1000
    x = rng.standard_normal(V) * 1.5
    x[:6] += 4.0
    T, k, p = 0.8, 20, 0.95
    _, d = sampler.sample_row(x, V, T, k, p, 0.0)
    keep = d["keep"]
    probs = d["q"][:keep] / d["q"][:keep].sum()
    n = 20000
    counts = {}
    for step in range(n):
        t, _ = sampler.sample_row(x, V, T, k, p, sampler.uniform(99, step, 0))
        counts[t] = counts.get(t, 0) + 1
    assert set(counts) <= set(d["order"][:keep].tolist())
    obs = np.array([counts.get(int(t), 0) for t in d["order"][:keep]], float)
    exp = probs * n
    chi2 = float(((obs - exp) ** 2 / exp).sum())
    dof = keep - 1
    # chi-square upper tail with dof degrees of freedom; Wilson-Hilferty normal approximation
    zscore = ((chi2 / dof) ** (1 / 3) - (1 - 2 / (9 * dof))) / math.sqrt(2 / (9 * dof))
    assert zscore < 3.5, (chi2, dof)


def test_q6_temperature():
    rng = np.random.default_rng(6)
    x = rng.standard_normal(300)
    _, d1 = sampler.sample_row(x, 300, 1.0, 20, 1.0, 0.5)
    _, d2 = sampler.sample_row(x, 300, 0.25, 20, 1.0, 0.5)
    assert np.array_equal(d1["order"], d2["order"])
    assert d2["q"][0] > d1["q"][0]
    # temperature T equals logits divided by T at temperature 1
    _, d3 = sampler.sample_row(x / 0.25, 300, 1.0, 20, 1.0, 0.5)
    np.testing.assert_allclose(d2["q"], d3["q"], rtol=1e-12)


def test_q7_draw_intervals_are_half_open():
    # Four equal logits: probabilities exactly 1/4, cumulative masses 1/4, 1/2,
    # 3/4, 1 (exact in binary, as are these 24-bit uniforms).
    x = np.zeros(4)
    for u, want in ((0.0, 0), (0.25 - 2.0 ** -24, 0), (0.25, 1), (0.5, 2), (0.75, 3), (1.0 - 2.0 ** -24, 3)):
        tok, d = sampler.sample_row(x, 4, 1.0, 4, 1.0, u)
        assert d["keep"] == 4 and tok == want, (u, tok)
    # With a top-p cut the same holds on the kept prefix's mass (1/2 here).
    for u, want in ((0.0, 0), (0.5, 1), (1.0 - 2.0 ** -24, 1)):
        tok, d = sampler.sample_row(x, 4, 1.0, 4, 0.5, u)
        assert d["keep"] == 2 and tok == want, (u, tok)


def test_bf16_rows_are_widened_exactly():
    x = np.array([1.0, -2.5, 3.25, 0.5], np.float32)
    bits = (x.view(np.uint32) >> 16).astype(np.uint16)
    assert sampler.sample_row(bits, 4, 0.8, 4, 1.0, 0.0)[0] == 2
