"""Pins of the oracle's gradient accumulation grad_theta += lambda s m (.) g~.

Central finite differences of a loss through the simulated state with the
draws held fixed (Eq. smat-gradient), the textbook add for s = keep = lambda
= 1 (torch's float32 add), zero gradient where a coordinate was dropped or
the scale is zero, and forward/backward mask identity.
"""
import numpy as np
import pytest
import torch

import oracle


def _rand(n, seed, scale=1.0):
    return (np.random.default_rng(seed).standard_normal(n) * scale).astype(np.float32)


@pytest.mark.parametrize("keep,rescale,s", [(0.5, 1, 0.6), (0.3, 0, 0.9), (1.0, 1, 0.25), (0.7, 1, 1.0)])
def test_finite_differences(keep, rescale, s):
    n = 48
    rng = np.random.default_rng(5)
    th = rng.standard_normal(n) * 0.02
    t0 = rng.standard_normal(n) * 0.02
    w = rng.standard_normal(n)
    p = dict(s=s, keep=keep, sigma=1e-3, rescale=rescale, noise_kind=0)
    key = (17, 3, 8)

    def loss(theta):
        y, _, _ = oracle.simulate_f64(theta, t0, "f64", p, *key)
        return float(np.sum(w * y) + 0.5 * np.sum(y * y))

    y, _, _ = oracle.simulate_f64(th, t0, "f64", p, *key)
    gsim = w + y                                   # dL/dtheta~
    h = 1e-6
    fd = np.empty(n)
    for k in range(n):
        e = np.zeros(n)
        e[k] = h
        fd[k] = (loss(th + e) - loss(th - e)) / (2 * h)
    got = oracle.backward_accum(gsim, "f64", np.zeros(n, dtype=np.float32), p, 1.0, *key)
    scale = np.abs(fd) + np.abs(gsim)
    assert np.all(np.abs(got - fd) <= 1e-6 * scale + 1e-12)


def test_textbook_add_when_everything_is_one():
    g = _rand(50000, 1, 1e-3)
    gs32 = _rand(50000, 2, 1e-2)
    p = dict(s=1.0, keep=1.0, sigma=0.0, rescale=1, noise_kind=0)
    got = oracle.backward_accum(gs32, "f32", g, p, 1.0, 1, 2, 3)
    want = (torch.from_numpy(g) + torch.from_numpy(gs32)).numpy()
    np.testing.assert_array_equal(got, want)
    gs16 = torch.from_numpy(gs32).to(torch.bfloat16)
    got16 = oracle.backward_accum(gs16.view(torch.int16).numpy().view(np.uint16), "bf16", g, p, 1.0, 1, 2, 3)
    want16 = (torch.from_numpy(g) + gs16.to(torch.float32)).numpy()
    np.testing.assert_array_equal(got16, want16)


def test_dropped_coordinates_unchanged_and_mask_matches_forward():
    n = 100000
    g = _rand(n, 3, 1e-3)
    gs = _rand(n, 4, 1e-2)
    p = dict(s=0.8, keep=0.3, sigma=1e-3, rescale=1, noise_kind=0)
    out = oracle.backward_accum(gs, "f32", g, p, 0.5, 9, 4, 2)
    _, kept, _ = oracle.simulate_f64(_rand(n, 5, 0.02), _rand(n, 6, 0.02), "f32", p, 9, 4, 2)
    np.testing.assert_array_equal(out.view(np.uint32)[~kept], g.view(np.uint32)[~kept])
    assert np.all(out[kept] != g[kept])          # g~ has no zeros, so every kept coordinate moves
    # kept coordinates moved by lambda * s / keep * g~ (to float32 rounding)
    coef = 0.5 * float(np.float32(0.8)) / float(np.float32(0.3))
    exact = g[kept].astype(np.float64) + coef * gs[kept].astype(np.float64)
    # one float32 rounding of the sum: half an ulp of the result, bounded via the operands
    bound = 2.0 ** -24 * np.abs(exact) + 1e-9 * (np.abs(g[kept]) + np.abs(coef * gs[kept]))
    assert np.all(np.abs(out[kept] - exact) <= bound)


def test_zero_scale_or_lambda_leaves_gradient():
    g = _rand(4000, 7, 1e-3)
    gs = _rand(4000, 8, 1e-2)
    for s, lam in ((0.0, 1.0), (0.9, 0.0)):
        p = dict(s=s, keep=0.5, sigma=0.0, rescale=1, noise_kind=0)
        np.testing.assert_array_equal(oracle.backward_accum(gs, "f32", g, p, lam, 1, 1, 1), g)


def test_all_dropped_leaves_gradient():
    g = _rand(4000, 9, 1e-3)
    p = dict(s=0.9, keep=0.0, sigma=1e-3, rescale=1, noise_kind=0)
    np.testing.assert_array_equal(oracle.backward_accum(_rand(4000, 10), "f32", g, p, 1.0, 1, 1, 1), g)


def test_invalid_lambda():
    with pytest.raises(ValueError):
        oracle.backward_accum(_rand(4, 1), "f32", _rand(4, 2), dict(s=1.0, keep=1.0, sigma=0.0), float("nan"), 0, 0, 0)
