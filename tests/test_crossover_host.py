"""Host arithmetic of the evicted-vs-full crossover (decode-compute analysis
of the appendix: evicted decode costs (1 + alpha) C_attn(B') per token, full
KV costs C_attn(l), so the two meet at l* = (1 + alpha) B' when C_attn is
proportional to l)."""
import pytest

from paper_2608_15797_amd.crossover import crossover_point, fit_line


def test_fit_line_recovers_an_exact_line():
    xs = [640, 1024, 2048, 4096, 8192]
    a, b = fit_line(xs, [0.25 + 3e-4 * x for x in xs])
    assert a == pytest.approx(0.25, abs=1e-12)
    assert b == pytest.approx(3e-4, rel=1e-12)


def test_fit_line_is_least_squares():
    # Residuals orthogonal to 1 and to x (they sum to 0, and so do x times
    # them) leave the least-squares line at y = 1 + 2x.
    xs = [0.0, 1.0, 2.0, 3.0]
    ys = [1.0 + 0.5, 3.0 - 0.5, 5.0 - 0.5, 7.0 + 0.5]
    a, b = fit_line(xs, ys)
    assert a == pytest.approx(1.0) and b == pytest.approx(2.0)


@pytest.mark.parametrize("alpha", [0.0, 0.25, 1.3])
def test_crossover_is_one_plus_alpha_times_b_prime_without_intercept(alpha):
    b, Bp = 2e-4, 640
    t = (1 + alpha) * b * Bp  # evicted cost per step
    best = {1024: b * 1024, 4096: b * 4096}
    r = crossover_point(t, 0.0, b, Bp, best)
    assert r["alpha"] == pytest.approx(alpha, abs=1e-3)
    assert r["ell_star"] == pytest.approx((1 + alpha) * Bp, abs=0.1)
    # Speed-up over full KV at l is l / l*.
    for k, v in r["speedup"].items():
        assert v == pytest.approx(int(k) / ((1 + alpha) * Bp), abs=1e-3)


def test_crossover_with_intercept():
    # t(l) = a + b l meets t at l* = (t - a) / b; alpha is measured at B'.
    a, b, Bp, t = 0.05, 1e-4, 640, 0.2
    r = crossover_point(t, a, b, Bp, {})
    assert r["ell_star"] == pytest.approx(1500.0, abs=0.1)
    assert r["alpha"] == pytest.approx(t / (a + b * Bp) - 1, abs=1e-3)
