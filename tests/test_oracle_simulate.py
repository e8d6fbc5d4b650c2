"""Pins of the oracle's simulated state theta~ = theta0 + s m (.) (theta - theta0) + eps.

Closed forms of Eq. smat-state (identity, all-dropped, zero scale), the
mean and variance of Prop. simulated-state-moments (including the rank-one
term from the shared scale), shard/offset invariance and argument errors.
"""
import math

import numpy as np
import pytest
import torch

import oracle


def _rand(n, seed, scale=0.02):
    return (np.random.default_rng(seed).standard_normal(n) * scale).astype(np.float32)


def _bf16_bits(x32):
    return torch.from_numpy(np.asarray(x32, dtype=np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


P = dict(s=0.7, keep=0.5, sigma=1e-3, rescale=1, noise_kind=0)


def test_identity_when_nothing_is_simulated():
    th = _rand(10000, 1)
    t0 = _rand(10000, 2)
    p = dict(s=1.0, keep=1.0, sigma=0.0, rescale=1, noise_kind=0)
    out32 = oracle.simulate(th, t0, "f32", "f32", p, 1, 2, 3)
    np.testing.assert_array_equal(out32, th)
    out16 = oracle.simulate(th, t0, "f32", "bf16", p, 1, 2, 3)
    np.testing.assert_array_equal(out16, _bf16_bits(th))   # torch's float32 -> bf16 rounding


def test_all_dropped_or_zero_scale_gives_base():
    th = _rand(5000, 3)
    t0_bits = _bf16_bits(_rand(5000, 4))
    for p in (dict(s=0.7, keep=0.0, sigma=0.0, rescale=1, noise_kind=0),
              dict(s=0.0, keep=0.3, sigma=0.0, rescale=1, noise_kind=0)):
        out = oracle.simulate(th, t0_bits, "bf16", "bf16", p, 5, 6, 7)
        np.testing.assert_array_equal(out, t0_bits)


def test_all_dropped_ignores_theta():
    t0 = _rand(5000, 5)
    p = dict(s=0.9, keep=0.0, sigma=2e-3, rescale=1, noise_kind=0)
    a = oracle.simulate(_rand(5000, 6), t0, "f32", "bf16", p, 1, 1, 1)
    b = oracle.simulate(_rand(5000, 7, 5.0), t0, "f32", "bf16", p, 1, 1, 1)
    np.testing.assert_array_equal(a, b)
    # and it differs from theta0 only by the noise: |theta~ - theta0| is a few sigma
    y, kept, eps = oracle.simulate_f64(_rand(5000, 6), t0, "f32", p, 1, 1, 1)
    assert not kept.any()
    np.testing.assert_allclose(y - t0.astype(np.float64), eps, rtol=0, atol=1e-17)
    assert np.abs(eps).max() < 6 * 2e-3


def test_kept_coordinates_move_by_scaled_task_vector():
    th = _rand(20000, 8)
    t0 = _rand(20000, 9)
    p = dict(s=0.6, keep=0.25, sigma=0.0, rescale=1, noise_kind=0)
    y, kept, _ = oracle.simulate_f64(th, t0, "f32", p, 3, 1, 2)
    d = th.astype(np.float64) - t0.astype(np.float64)
    t = np.float32(0.6) / np.float32(0.25)   # alpha / keep, here exactly 2.4 in float32 terms
    np.testing.assert_allclose(y[kept] - t0[kept], float(np.float32(0.6)) / float(np.float32(0.25)) * d[kept],
                               rtol=1e-12, atol=1e-18)
    np.testing.assert_array_equal(y[~kept], t0[~kept].astype(np.float64))
    assert abs(float(t) - 2.4) < 1e-6


@pytest.mark.parametrize("keep,rescale", [(0.5, 1), (0.2, 1), (0.2, 0), (1.0, 1)])
def test_moments_fixed_scale(keep, rescale):
    # Delta == c everywhere, one s: E[theta~] = theta0 + s c (E[m] = 1 with rescale, keep without);
    # Var = s^2 c^2 Var(m) + sigma^2 (Prop. simulated-state-moments with v_alpha = 0)
    n = 1 << 20
    c, s, sigma = 3e-3, 0.7, 1e-3
    t0 = np.zeros(n, dtype=np.float32)
    th = np.full(n, c, dtype=np.float32)
    p = dict(s=s, keep=keep, sigma=sigma, rescale=rescale, noise_kind=0)
    y, _, _ = oracle.simulate_f64(th, t0, "f32", p, 21, 0, 0)
    k = float(np.float32(keep))
    cc, ss = float(np.float32(c)), float(np.float32(s))
    if rescale:
        mean_m, var_m = 1.0, (1 - k) / k
    else:
        mean_m, var_m = k, k * (1 - k)
    want_mean = ss * cc * mean_m
    want_var = ss ** 2 * cc ** 2 * var_m + float(np.float32(sigma)) ** 2
    d = y
    assert abs(d.mean() - want_mean) <= 5 * math.sqrt(want_var / n)
    m4 = np.mean((d - d.mean()) ** 4)
    assert abs(d.var() - want_var) <= 5 * math.sqrt(max(m4 - want_var ** 2, 1e-40) / n)


def test_moments_random_scale_rank_one_term():
    # alpha ~ U[alpha_min, 1] shared by all coordinates of a step: the per-step mean
    # of theta~ - theta0 over coordinates has variance v_alpha c^2 + (s_alpha c^2 (1-q)/q + sigma^2)/n
    # and overall mean alpha_bar c (Prop. simulated-state-moments).
    n, steps, amin, keep, sigma, c = 512, 2000, 0.2, 0.5, 1e-3, 2e-3
    rng = np.random.default_rng(77)
    alphas = rng.uniform(amin, 1.0, size=steps).astype(np.float32)
    t0 = np.zeros(n, dtype=np.float32)
    th = np.full(n, c, dtype=np.float32)
    means = np.empty(steps)
    for i, a in enumerate(alphas):
        y, _, _ = oracle.simulate_f64(th, t0, "f32", dict(s=float(a), keep=keep, sigma=sigma, rescale=1), 5, i, 0)
        means[i] = y.mean()
    cc = float(np.float32(c))
    abar = (1 + amin) / 2
    v_a = (1 - amin) ** 2 / 12
    s_a = abar ** 2 + v_a
    q = keep
    per_coord = s_a * cc ** 2 * (1 - q) / q + sigma ** 2
    want_var = v_a * cc ** 2 + per_coord / n
    assert abs(means.mean() - abar * cc) <= 5 * math.sqrt(want_var / steps)
    # variance of a sample variance of a near-uniform mixture: allow 5 SE using its kurtosis
    m4 = np.mean((means - means.mean()) ** 4)
    assert abs(means.var() - want_var) <= 5 * math.sqrt((m4 - means.var() ** 2) / steps)
    # and it is dominated by the shared-scale term, not by the per-coordinate terms
    assert means.var() > 0.8 * v_a * cc ** 2


def test_shard_offsets_reproduce_whole_tensor():
    th = _rand(3001, 10)
    t0 = _bf16_bits(_rand(3001, 11))
    full = oracle.simulate(th, t0, "bf16", "bf16", P, 4, 8, 12, 0)
    for cut in (1, 4, 1000, 1003, 3000):
        a = oracle.simulate(th[:cut], t0[:cut], "bf16", "bf16", P, 4, 8, 12, 0)
        b = oracle.simulate(th[cut:], t0[cut:], "bf16", "bf16", P, 4, 8, 12, cut)
        np.testing.assert_array_equal(np.concatenate([a, b]), full)


def test_multi_list_matches_single_calls():
    ths = [_rand(n, 20 + n) for n in (1, 7, 100, 4099)]
    t0s = [_bf16_bits(_rand(n, 30 + n)) for n in (1, 7, 100, 4099)]
    ps = [dict(P, s=0.3 + 0.1 * i) for i in range(4)]
    outs = oracle.simulate_multi(ths, t0s, "bf16", "bf16", ps, 9, 2, [5, 1, 9, 2])
    for i in range(4):
        np.testing.assert_array_equal(outs[i], oracle.simulate(ths[i], t0s[i], "bf16", "bf16", ps[i], 9, 2, [5, 1, 9, 2][i]))
    with pytest.raises(ValueError):
        oracle.simulate_multi(ths[:2], t0s[:2], "bf16", "bf16", ps[:2], 9, 2, [3, 3])


@pytest.mark.parametrize("bad", [dict(keep=1.5), dict(keep=-0.1), dict(sigma=-1e-3), dict(sigma=float("nan")),
                                 dict(s=float("inf")), dict(keep=float("nan")), dict(noise_kind=7)])
def test_invalid_arguments(bad):
    p = dict(P, **bad)
    with pytest.raises(ValueError):
        oracle.simulate(_rand(8, 1), _rand(8, 2), "f32", "f32", p, 0, 0, 0)
