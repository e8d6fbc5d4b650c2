"""The theta~ bar of the GPU tests (tests/tolerances.py) against the kernel's fp32 arithmetic
emulated exactly on the CPU: t = fl32(s/keep), a = fma(-t, theta0, theta0), b = fma(t, theta, a),
c = fma(sigma, z', b) with a Box-Muller value z' within Z_TOL of the exact one, then one rounding to
the output type.  Each fma is one rounding of the exact a*b + c, formed in 80-bit extended
precision (the product of two fp32 values is exact there, and rounding a 64-bit-significand value to
fp32 is innocuous double rounding), so the emulation gives the kernel's bits up to z'.  Every
element must pass, with a bf16 output the 1-ulp ("strict") elements must be all but a few per
thousand, and the
lerp's inner rounding must really exceed the 2^-22 (|theta0| + |t D| + |eps|) form for large t."""
import numpy as np
import pytest

import oracle
from tolerances import U, Z_TOL, check_theta_tilde, ordered, theta_tilde_bound

LD = np.longdouble


def fma32(a, b, c):
    return (LD(1) * np.asarray(a, np.float32).astype(LD) * np.asarray(b, np.float32).astype(LD)
            + np.asarray(c, np.float32).astype(LD)).astype(np.float32)


def kernel_simulate(th, t0_bits, p, kept, z_dev, out_dtype):
    t0 = oracle.bf16_bits_to_f64(t0_bits).astype(np.float32)
    s32, k32 = np.float32(p["s"]), np.float32(p["keep"])
    t = np.float32(float(s32) / float(k32)) if (p["rescale"] and 0 < k32 < 1) else s32
    lerp = fma32(np.full_like(th, t), th, fma32(np.full_like(th, -t), t0, t0))
    y = np.where(kept, lerp, t0)
    if p["sigma"] > 0:
        y = fma32(np.full_like(th, np.float32(p["sigma"])), z_dev, y)
    return oracle.round_to(y.astype(np.float64), out_dtype) if out_dtype == "bf16" else y


@pytest.mark.parametrize("s,keep,rescale,sigma", [(0.7, 0.5, 1, 1e-3), (1.0, 0.1, 1, 3e-4), (0.93, 0.1, 1, 0.0),
                                                  (0.3, 1.0, 1, 2e-4), (1.0, 1.0, 0, 0.0), (0.55, 0.2, 0, 1e-4),
                                                  (1.0, 0.11, 1, 5e-5)])
@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_bound_contains_the_kernel_arithmetic(s, keep, rescale, sigma, out_dtype):
    rng = np.random.default_rng(int(s * 1000) + int(keep * 100) + rescale)
    n = 1 << 16
    t0_bits = oracle.round_to_bf16_bits(rng.standard_normal(n) * 0.02)
    th = (oracle.bf16_bits_to_f64(t0_bits) + rng.standard_normal(n) * 2e-4).astype(np.float32)
    th[:64] = -oracle.bf16_bits_to_f64(t0_bits[:64]).astype(np.float32)     # theta = -theta0: large D
    p = dict(s=s, keep=keep, rescale=rescale, sigma=sigma, noise_kind=0)
    y, kept, eps = oracle.simulate_f64(th, t0_bits, "bf16", p, 7, 3, 1)
    z = oracle.gaussian_z(7, 3, 1, 0, n)
    z_dev = (z + rng.uniform(-Z_TOL, Z_TOL, n) * 0.999).astype(np.float32)
    got = kernel_simulate(th, t0_bits, p, kept, z_dev, out_dtype)
    coef = np.where(kept, oracle.coefficient(s, keep, rescale), 0.0)
    ok, strict = check_theta_tilde(got, out_dtype, y, th, oracle.bf16_bits_to_f64(t0_bits), coef, eps, np.float32(sigma))
    assert ok.all(), np.flatnonzero(~ok)[:5]
    if out_dtype == "bf16":
        # an fp32 error of a few u is far below half a bf16 ulp except near zero results; an fp32
        # output is held to the absolute bound everywhere
        assert (~strict).mean() <= 1e-3
        assert np.abs(ordered(got) - ordered(oracle.round_to_bf16_bits(y)))[strict].max(initial=0) <= 1


def test_two_fma_lerp_needs_the_theta0_term_for_large_t():
    """At t = 10 (keep 0.1 rescaled) the inner fma's rounding, u |theta0| |1 - t|, exceeds a bound of
    the form 4u (|theta0| + |t D| + |eps|) on some elements: the bar cannot take that form."""
    rng = np.random.default_rng(5)
    n = 1 << 16
    t0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
    th = (t0 + rng.standard_normal(n) * 2e-4).astype(np.float32)
    t = np.float32(10.0)
    c = fma32(np.full(n, t), th, fma32(np.full(n, -t), t0, t0)).astype(np.float64)
    y = t0.astype(np.float64) + 10.0 * (th.astype(np.float64) - t0.astype(np.float64))
    err = np.abs(c - y)
    no_theta0_term = 4 * U * (np.abs(t0) + 10.0 * np.abs(th.astype(np.float64) - t0))
    assert (err > no_theta0_term).any()
    assert (err <= theta_tilde_bound(th.astype(np.float64), t0.astype(np.float64), 10.0, 0.0, 0.0)).all()


def test_nonstrict_cap_allowance_is_a_poisson_tail():
    """The small-tensor allowance of the non-strict cap: at the cap's own rate (one element per
    1,000) a 1,000-element tensor reaches the allowance + 1 with probability about 1e-6, and the cap
    is the larger of the allowance and the 1e-3 fraction."""
    from scipy.stats import poisson

    from tolerances import NONSTRICT_MAX_FRACTION, NONSTRICT_SMALL_ALLOWANCE, nonstrict_within_cap

    tail = poisson.sf(NONSTRICT_SMALL_ALLOWANCE, NONSTRICT_MAX_FRACTION * 1000)
    assert 1e-7 < tail < 2e-6
    assert nonstrict_within_cap(8, 1042) and not nonstrict_within_cap(9, 1042)
    assert nonstrict_within_cap(1000, 10 ** 6) and not nonstrict_within_cap(1001, 10 ** 6)
    assert nonstrict_within_cap(0, 0)
