"""Pins of the oracle's N-expert merge (Eq. merged-state): weight averaging is the mean of the
experts, Task Arithmetic is theta0 + gamma * sum of task vectors, one expert reproduces the
simulated state without noise, DARE masks are the training masks of each expert's (seed, step)
and unbiased (E[m] = 1), and the result does not depend on the order of the experts."""
import math

import numpy as np
import pytest

import oracle

N_EL = 4099


def experts(n_exp, seed=0, n=N_EL):
    rng = np.random.default_rng(seed)
    theta0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
    ex = [(theta0 + rng.standard_normal(n) * 1e-3).astype(np.float32) for _ in range(n_exp)]
    return theta0, ex


def term(gamma, keep=1.0, seed=1, step=0, rescale=1):
    return dict(gamma=gamma, keep=keep, rescale=rescale, seed=seed, step=step)


@pytest.mark.parametrize("n_exp", [2, 4, 8])
def test_weight_averaging_is_the_mean(n_exp):
    theta0, ex = experts(n_exp)
    y = oracle.merge_f64(ex, "f32", theta0, "f32", [term(1.0 / n_exp)] * n_exp, 3)   # 1/N exact in fp32
    np.testing.assert_allclose(y, np.mean(np.stack(ex).astype(np.float64), axis=0), rtol=0, atol=1e-15)


def test_task_arithmetic_closed_form():
    theta0, ex = experts(7, 1)
    g = 0.3
    y = oracle.merge_f64(ex, "f32", theta0, "f32", [term(g)] * 7, 5)
    g32 = float(np.float32(g))
    want = theta0.astype(np.float64) + g32 * np.sum(np.stack(ex).astype(np.float64) - theta0.astype(np.float64), axis=0)
    np.testing.assert_allclose(y, want, rtol=0, atol=1e-15)


@pytest.mark.parametrize("keep,rescale", [(0.5, 1), (0.3, 0), (1.0, 1), (0.0, 1)])
def test_one_expert_is_the_simulated_state_without_noise(keep, rescale):
    theta0, (th,) = experts(1, 2)
    t0_bits = oracle.round_to_bf16_bits(theta0.astype(np.float64))
    y = oracle.merge_f64([th], "f32", t0_bits, "bf16", [term(0.6, keep, seed=77, step=12, rescale=rescale)], 9, 40)
    ys, _, _ = oracle.simulate_f64(th, t0_bits, "bf16", dict(s=0.6, keep=keep, sigma=0.0, rescale=rescale), 77, 12, 9, 40)
    np.testing.assert_array_equal(y, ys)


def test_dare_masks_are_each_experts_training_masks():
    theta0, ex = experts(3, 3)
    terms = [term(0.5, 0.3, seed=10 + j, step=4 + j) for j in range(3)]
    y = oracle.merge_f64(ex, "f32", theta0, "f32", terms, 2, 8)
    t0 = theta0.astype(np.float64)
    want = t0.copy()
    for x, t in zip(ex, terms):
        kept = oracle.keep_mask(t["seed"], t["step"], 2, 8, N_EL, t["keep"])
        k32 = float(np.float32(t["keep"]))
        want += np.where(kept, float(np.float32(0.5)) / k32 * (x.astype(np.float64) - t0), 0.0)
    np.testing.assert_allclose(y, want, rtol=0, atol=1e-15)
    # an expert with keep = 0 contributes nothing
    y0 = oracle.merge_f64(ex + [ex[0] * 3], "f32", theta0, "f32", terms + [term(5.0, 0.0)], 2, 8)
    np.testing.assert_array_equal(y0, y)


def test_dare_merge_is_unbiased():
    # E[m] = 1 per coordinate, so averaging over seeds gives Task Arithmetic; the aggregate error
    # over all coordinates is checked against the exact variance gamma^2 sum_j Delta_j^2 (1 - k)/k
    theta0, ex = experts(3, 4, n=2048)
    g, keep, S = 0.4, 0.3, 200
    t0 = theta0.astype(np.float64)
    ta = oracle.merge_f64(ex, "f32", theta0, "f32", [term(g)] * 3, 1)
    acc = np.zeros_like(t0)
    for s in range(S):
        acc += oracle.merge_f64(ex, "f32", theta0, "f32", [term(g, keep, seed=1000 * s + j) for j in range(3)], 1)
    dev = acc / S - ta
    k32 = float(np.float32(keep))
    var = float(np.float32(g)) ** 2 * sum((x.astype(np.float64) - t0) ** 2 for x in ex) * (1 - k32) / k32 / S
    z = np.sum(dev) / math.sqrt(np.sum(var))          # a sum of independent zero-mean deviations
    assert abs(z) < 5
    assert 0.5 < np.mean(dev ** 2) / np.mean(var) < 1.5


def test_order_of_experts_does_not_matter():
    theta0, ex = experts(5, 5)
    terms = [term(0.2 + 0.1 * j, 0.5 + 0.1 * j, seed=j, step=j) for j in range(5)]
    y = oracle.merge_f64(ex, "f32", theta0, "f32", terms, 6)
    perm = [3, 0, 4, 2, 1]
    yp = oracle.merge_f64([ex[i] for i in perm], "f32", theta0, "f32", [terms[i] for i in perm], 6)
    np.testing.assert_allclose(yp, y, rtol=0, atol=1e-16)


def test_rounding_and_errors():
    theta0, ex = experts(2, 6)
    out = oracle.merge(ex, "f32", theta0, "f32", "bf16", [term(0.5)] * 2, 0)
    assert out.dtype == np.uint16
    np.testing.assert_array_equal(out, oracle.round_to_bf16_bits(oracle.merge_f64(ex, "f32", theta0, "f32",
                                                                                   [term(0.5)] * 2, 0)))
    with pytest.raises(ValueError):
        oracle.merge_f64(ex, "f32", theta0, "f32", [term(0.5)], 0)              # one term per expert
    with pytest.raises(ValueError):
        oracle.merge_f64(ex, "f32", theta0, "f32", [term(0.5, keep=1.5)] * 2, 0)
    with pytest.raises(ValueError):
        oracle.merge_f64(ex, "f32", theta0, "f32", [term(float("nan"))] * 2, 0)
