"""Pins of the oracle's gradient norm and clipping factor, the inputs of norm clipping ahead of the
fused optimizer step.  Checked against NumPy's norm, kept-coordinate counts of the pinned mask,
and PyTorch's own torch.nn.utils.clip_grad_norm_ on the materialised gradient (CPU, float64)."""
import math

import numpy as np
import pytest
import torch

import oracle

SEED, STEP = 0xC11F, 7


def test_unmasked_norm_is_the_plain_l2_norm():
    rng = np.random.default_rng(1)
    g = (rng.standard_normal(5000) * 1e-2).astype(np.float32)
    p = dict(s=1.0, keep=1.0, sigma=0.0, rescale=1)
    sq = oracle.grad_sqnorm(g, "f32", p, 1.0, SEED, STEP, 0)
    assert math.isclose(math.sqrt(sq), float(np.linalg.norm(g.astype(np.float64))), rel_tol=1e-13)


@pytest.mark.parametrize("rescale", [0, 1])
def test_unit_gradient_counts_kept_coordinates(rescale):
    n, keep = 200_003, 0.3
    ones = np.ones(n, np.float32)
    p = dict(s=1.0, keep=keep, sigma=0.0, rescale=rescale)
    kept = int(oracle.keep_mask(SEED, STEP, 4, 0, n, keep).sum())
    sq = oracle.grad_sqnorm(ones, "f32", p, 1.0, SEED, STEP, 4)
    k32 = float(np.float32(keep))                   # keep enters as its fp32 value, as at the C ABI
    assert sq == pytest.approx(kept / (k32 * k32 if rescale else 1.0), rel=1e-13)
    assert abs(kept - keep * n) < 5 * math.sqrt(n * keep * (1 - keep))      # binomial, 5 sigma


def test_scaling_in_lambda_and_alpha():
    rng = np.random.default_rng(2)
    g = (rng.standard_normal(3001) * 1e-2).astype(np.float32)
    p = dict(s=0.5, keep=0.5, sigma=0.0, rescale=1)
    base = oracle.grad_sqnorm(g, "f32", p, 1.0, SEED, STEP, 1)
    assert oracle.grad_sqnorm(g, "f32", p, 2.0, SEED, STEP, 1) == pytest.approx(4 * base, rel=1e-14)
    assert oracle.grad_sqnorm(g, "f32", dict(p, s=0.25), 1.0, SEED, STEP, 1) == pytest.approx(base / 4, rel=1e-14)
    assert oracle.grad_sqnorm(g, "f32", dict(p, keep=0.0), 1.0, SEED, STEP, 1) == 0.0     # all dropped


def test_shards_add_up_to_the_whole_tensor():
    rng = np.random.default_rng(3)
    n, cut = 10_007, 4_093
    g = (rng.standard_normal(n) * 1e-2).astype(np.float32)
    acc = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    p = dict(s=0.8, keep=0.4, sigma=0.0, rescale=1)
    whole = oracle.grad_sqnorm(g, "f32", p, 0.5, SEED, STEP, 9, grad_acc=acc)
    parts = oracle.grad_sqnorm_multi([g[:cut], g[cut:]], "f32", [p, p], 0.5, SEED, STEP, [9, 9], [0, cut],
                                     grad_accs=[acc[:cut], acc[cut:]])
    assert parts == pytest.approx(whole, rel=1e-13)


@pytest.mark.parametrize("max_norm", [1e-3, 1.0, 1e6])
def test_clipping_matches_torch_clip_grad_norm(max_norm):
    rng = np.random.default_rng(4)
    sizes = [1000, 37, 4096]
    gs = [(rng.standard_normal(n) * 5e-3).astype(np.float32) for n in sizes]
    accs = [(rng.standard_normal(n) * 1e-3).astype(np.float32) for n in sizes]
    params = [dict(s=0.6, keep=0.5, sigma=1e-3, rescale=1), dict(s=0.6, keep=1.0, sigma=0.0, rescale=1),
              dict(s=0.6, keep=0.2, sigma=0.0, rescale=0)]
    ids = [0, 1, 2]
    for use_acc in (False, True):
        acc = accs if use_acc else None
        sq = oracle.grad_sqnorm_multi(gs, "f32", params, 0.5, SEED, STEP, ids, grad_accs=acc)
        coef = oracle.clip_coefficient(math.sqrt(sq), max_norm)
        grads = [oracle.simulated_gradient(gs[i], "f32", params[i], 0.5, SEED, STEP, ids[i], 0,
                                           None if acc is None else acc[i]) for i in range(3)]
        tparams = []
        for g in grads:
            t = torch.nn.Parameter(torch.zeros(g.size, dtype=torch.float64))
            t.grad = torch.from_numpy(g.copy())
            tparams.append(t)
        total = float(torch.nn.utils.clip_grad_norm_(tparams, max_norm, foreach=False))
        assert total == pytest.approx(math.sqrt(sq), rel=1e-13)
        for t, g in zip(tparams, grads):
            np.testing.assert_allclose(t.grad.numpy(), coef * g, rtol=1e-13, atol=0)
        assert (coef < 1.0) == (max_norm < total)


@pytest.mark.parametrize("bad", [0.0, -1.0, float("nan"), float("inf")])
def test_clip_rejects_bad_max_norm(bad):
    with pytest.raises(ValueError):
        oracle.clip_coefficient(1.0, bad)
