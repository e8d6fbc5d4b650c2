"""Pins of the oracle's fused optimizer step: the AdamW definition against PyTorch's own AdamW
(CPU, float64) over several steps; Adam's first-step magnitude; zero gradient on dropped
coordinates entering the update; argument errors."""

import numpy as np
import pytest
import torch

import oracle

HP = dict(lr=2e-5, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-3, grad_scale=1.0, step=1)


@pytest.mark.parametrize("wd", [0.0, 1e-3, 0.1])
def test_matches_torch_adamw_over_steps(wd):
    rng = np.random.default_rng(3)
    n = 1000
    theta = rng.standard_normal(n) * 0.02
    param = torch.nn.Parameter(torch.from_numpy(theta.copy()))
    hp = dict(HP, weight_decay=wd, lr=1e-3)
    opt = torch.optim.AdamW([param], lr=float(np.float32(hp["lr"])), betas=(float(np.float32(0.9)), float(np.float32(0.999))),
                            eps=float(np.float32(1e-8)), weight_decay=float(np.float32(wd)), foreach=False)
    th, m1, m2 = theta.copy(), np.zeros(n), np.zeros(n)
    for k in range(1, 6):
        g = rng.standard_normal(n) * 1e-2
        param.grad = torch.from_numpy(g.copy())
        opt.step()
        th, m1, m2 = oracle.adamw_update(th, m1, m2, g, dict(hp, step=k))
        st = opt.state[param]
        np.testing.assert_allclose(th, param.detach().numpy(), rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(m1, st["exp_avg"].numpy(), rtol=1e-12, atol=1e-18)
        np.testing.assert_allclose(m2, st["exp_avg_sq"].numpy(), rtol=1e-12, atol=1e-22)


def test_first_step_is_lr_sized():
    # from zero moments, Adam's first step is lr * g / (|g| + eps) (bias correction undoes (1 - beta))
    g = np.array([1e-2, -3e-3, 5e-1, -2.0])
    th, m1, m2 = oracle.adamw_update(np.zeros(4), np.zeros(4), np.zeros(4), g, dict(HP, weight_decay=0.0))
    np.testing.assert_allclose(th, -float(np.float32(2e-5)) * g / (np.abs(g) + float(np.float32(1e-8))), rtol=1e-9)


def test_simulated_gradient_and_dropped_coordinates():
    rng = np.random.default_rng(4)
    n = 4096
    gs = (rng.standard_normal(n) * 1e-2).astype(np.float32)
    acc = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    p = dict(s=0.7, keep=0.25, sigma=1e-3, rescale=1)
    kept = oracle.keep_mask(5, 3, 1, 0, n, 0.25)
    g = oracle.simulated_gradient(gs, "f32", p, 0.5, 5, 3, 1)
    assert np.all(g[~kept] == 0.0)
    np.testing.assert_allclose(g[kept], 0.5 * float(np.float32(0.7)) / 0.25 * gs[kept].astype(np.float64), rtol=1e-14)
    # with an accumulated gradient, dropped coordinates carry it unchanged; grad_scale multiplies all
    g2 = oracle.simulated_gradient(gs, "f32", p, 0.5, 5, 3, 1, grad_acc=acc, grad_scale=0.5)
    np.testing.assert_allclose(g2[~kept], 0.5 * acc[~kept].astype(np.float64), rtol=1e-15)
    # the fused step equals the backward accumulation followed by the AdamW definition
    th = (rng.standard_normal(n) * 0.02).astype(np.float32)
    (t1, _, _), _ = oracle.adamw_fused(gs, "f32", th, np.zeros(n), np.zeros(n), p, 0.5, HP, 5, 3, 1, grad_acc=acc)
    gacc = oracle.backward_accum(gs, "f32", acc, p, 0.5, 5, 3, 1)
    t2, _, _ = oracle.adamw_update(th, np.zeros(n), np.zeros(n), gacc.astype(np.float64), HP)
    np.testing.assert_allclose(t1, t2, rtol=1e-6, atol=1e-12)


@pytest.mark.parametrize("bad", [dict(beta1=1.0), dict(beta2=-0.1), dict(eps=0.0), dict(lr=float("nan")),
                                 dict(step=0), dict(weight_decay=-1.0), dict(grad_scale=float("inf"))])
def test_invalid_hyperparameters(bad):
    with pytest.raises(ValueError):
        oracle.adamw_update(np.zeros(2), np.zeros(2), np.zeros(2), np.zeros(2), dict(HP, **bad))
