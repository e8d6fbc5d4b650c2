"""Pins of the oracle's scale draw (oracle.scale_draw): the shared scale alpha ~ U[alpha_min, 1] of
one simulated update (Sec. 4.1, "Scale") as a function of (seed, step).  Checked against the
Philox bijection itself (pinned by its known-answer vectors), the closed forms at alpha_min = 0 and
1, the range, the law (Kolmogorov-Smirnov against U[alpha_min, 1], and the mean), and that the
draw depends on the seed and the step."""
import numpy as np
import pytest
from scipy import stats

import oracle


def test_alpha_min_zero_is_the_24_bit_uniform():
    # alpha_min = 0: alpha = (w0 >> 8) 2^-24 exactly, w0 = word 0 of counter (0, 0, 0, 4 step + 2)
    seed = 0x0123456789ABCDEF
    for step in (0, 1, 7, 12345, 2 ** 30 - 1):
        w = oracle.philox4x32(0, 0, 0, 4 * step + 2, seed & 0xFFFFFFFF, seed >> 32)
        want = (int(w[0]) >> 8) / 2.0 ** 24
        assert oracle.scale_draw(seed, step, 0.0) == want


def test_alpha_min_one_is_one():
    assert all(oracle.scale_draw(9, s, 1.0) == 1.0 for s in range(50))


@pytest.mark.parametrize("alpha_min", [0.2, 0.1, 0.75])
def test_range_law_and_mean(alpha_min):
    n = 20000
    a = np.array([oracle.scale_draw(77, s, alpha_min) for s in range(n)])
    lo = float(np.float32(alpha_min))
    assert a.min() >= lo and a.max() <= 1.0
    assert stats.kstest(a, "uniform", args=(lo, 1.0 - lo)).pvalue > 1e-3
    sd = (1.0 - lo) / np.sqrt(12.0 * n)
    assert abs(a.mean() - (1.0 + lo) / 2.0) < 5 * sd
    # every value is the fp32 rounding of lo + (1 - lo) u for a 24-bit u
    assert np.all(a.astype(np.float32).astype(np.float64) == a)


def test_depends_on_seed_and_step_only():
    x = [oracle.scale_draw(5, s, 0.2) for s in range(200)]
    assert x == [oracle.scale_draw(5, s, 0.2) for s in range(200)]
    y = [oracle.scale_draw(6, s, 0.2) for s in range(200)]
    assert sum(a == b for a, b in zip(x, y)) < 5
    assert len(set(x)) > 190
    with pytest.raises(ValueError):
        oracle.scale_draw(5, 0, 1.5)
