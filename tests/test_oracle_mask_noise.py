"""Pins of the oracle's mask and noise draws.

Mask (Eq. smat-mask): keep-rate within binomial bounds, E[m] = 1 and
E[m^2] = 1/keep with the 1/keep rescale (Prop. simulated-state-moments,
proof), degenerate keep values, independence across steps/tensors/streams.
Noise (Sec. 4.1, "Perturb"; Box-Muller): zero mean, unit variance, a KS test
against N(0, 1), closed-form special values and the pairing invariant.
"""
import math

import numpy as np
import pytest
from scipy import stats

import oracle

N = 1 << 20


@pytest.mark.parametrize("keep", [0.1, 0.2, 0.5, 0.9, 0.123456])
def test_keep_rate_binomial(keep):
    kept = oracle.keep_mask(11, 3, 7, 0, N, keep)
    q = oracle.mask_threshold(keep) / 2.0 ** 32
    assert abs(q - float(np.float32(keep))) <= 2.0 ** -32
    assert abs(kept.mean() - q) <= 5 * math.sqrt(q * (1 - q) / N)


@pytest.mark.parametrize("keep", [0.1, 0.5, 0.8])
def test_mask_moments(keep):
    kept = oracle.keep_mask(12, 0, 1, 0, N, keep)
    m = oracle.mask_values(kept, keep, True)
    k = float(np.float32(keep))
    # E[m] = 1, E[m^2] = 1/keep; standard errors from the two-point distribution
    se1 = math.sqrt((1 / k - 1) / N)
    assert abs(m.mean() - 1.0) <= 5 * se1
    var_m2 = (1 / k ** 3) - (1 / k) ** 2
    assert abs((m ** 2).mean() - 1 / k) <= 5 * math.sqrt(var_m2 / N)
    # without rescale the kept value is 1 and E[m] = keep
    m0 = oracle.mask_values(kept, keep, False)
    assert set(np.unique(m0)) <= {0.0, 1.0}


def test_mask_degenerate_keeps():
    assert oracle.keep_mask(1, 2, 3, 0, 1000, 1.0).all()
    assert not oracle.keep_mask(1, 2, 3, 0, 1000, 0.0).any()
    assert oracle.mask_threshold(1.0) is None and oracle.mask_threshold(0.0) is None
    assert oracle.mask_threshold(0.5) == 2 ** 31
    # keep = 0.5 keeps exactly the words whose top bit is clear
    w = oracle.element_words(1, 2, 3, 0, 4096, oracle.STREAM_MASK)
    np.testing.assert_array_equal(oracle.keep_mask(1, 2, 3, 0, 4096, 0.5), (w >> 31) == 0)
    # the largest float32 below 1 still draws and keeps almost everything
    k = float(np.nextafter(np.float32(1.0), np.float32(0.0)))
    assert oracle.mask_threshold(k) == 2 ** 32 - 2 ** 8


def test_mask_independence():
    n = 1 << 18
    a = oracle.keep_mask(5, 10, 2, 0, n, 0.5).astype(np.float64)
    others = [oracle.keep_mask(5, 11, 2, 0, n, 0.5),
              oracle.keep_mask(5, 10, 3, 0, n, 0.5),
              oracle.keep_mask(6, 10, 2, 0, n, 0.5),
              oracle.keep_mask(5, 10, 2, 1, n, 0.5)]   # shifted by one element
    for b in others:
        rho = np.corrcoef(a, b.astype(np.float64))[0, 1]
        assert abs(rho) <= 5 / math.sqrt(n)
    # the mask stream is independent of the noise stream at the same counter
    z = oracle.gaussian_z(5, 10, 2, 0, n)
    assert abs(np.corrcoef(a, z)[0, 1]) <= 5 / math.sqrt(n)


def test_gaussian_moments_and_ks():
    z = oracle.gaussian_z(0x5EED0000, 0, 0, 0, N)
    assert abs(z.mean()) <= 5 / math.sqrt(N)
    assert abs(z.var() - 1.0) <= 5 * math.sqrt(2.0 / N)
    assert stats.kstest(z, "norm").pvalue > 1e-4
    # each lane on its own is standard normal too (pairing does not bias a lane)
    for lane in range(4):
        zl = z[lane::4]
        assert abs(zl.mean()) <= 5 / math.sqrt(zl.size)
        assert abs(zl.var() - 1.0) <= 5 * math.sqrt(2.0 / zl.size)
    # neighbouring lanes are uncorrelated
    assert abs(np.corrcoef(z[0::4], z[1::4])[0, 1]) <= 5 / math.sqrt(N / 4)
    assert abs(np.corrcoef(z[1::4], z[2::4])[0, 1]) <= 5 / math.sqrt(N / 4)


def test_box_muller_special_values():
    # u1 = 1 (top 24 bits all ones) gives r = 0
    zc, zs = oracle.box_muller(np.array([0xFFFFFFFF, 0xFFFFFF00]), np.array([0x12345678, 0]))
    assert np.all(zc == 0.0) and np.all(zs == 0.0)
    # u1 = 1/2, u2 = 0: (sqrt(2 ln 2), 0); u2 = 1/4: (~0, sqrt(2 ln 2)); u2 = 1/2: (-sqrt(2 ln 2), ~0)
    a = np.array([(2 ** 23 - 1) << 8] * 3, dtype=np.uint64)
    b = np.array([0, 2 ** 30, 2 ** 31], dtype=np.uint64)
    zc, zs = oracle.box_muller(a, b)
    r = math.sqrt(2 * math.log(2))
    np.testing.assert_allclose(zc, [r, 0.0, -r], atol=1e-15)
    np.testing.assert_allclose(zs, [0.0, r, 0.0], atol=1e-15)
    # low 8 bits of either word are ignored (24-bit uniforms)
    zc2, zs2 = oracle.box_muller(a | np.uint64(0xFF), b | np.uint64(0x7F))
    np.testing.assert_array_equal(zc, zc2)
    np.testing.assert_array_equal(zs, zs2)


def test_gaussian_pairing_invariant():
    # lanes 0,1 of a group share u1 from word 0; lanes 2,3 share u1 from word 2:
    # z0^2 + z1^2 = -2 ln u1(w0) and z2^2 + z3^2 = -2 ln u1(w2); the sine lane is
    # non-negative exactly when u2 < 1/2 (top bit of its word clear)
    n = 4096
    z = oracle.gaussian_z(9, 1, 4, 0, n)
    w = oracle.group_words(9, 1, 4, np.arange(n // 4), oracle.STREAM_NOISE)
    for pair in (0, 2):
        u1 = ((w[pair].astype(np.float64) // 256) + 1) / 2.0 ** 24
        r2 = z[pair::4] ** 2 + z[pair + 1::4] ** 2
        np.testing.assert_allclose(r2, -2 * np.log(u1), rtol=1e-12, atol=1e-15)
        top = (w[pair + 1] >> 31) == 0
        assert np.all((z[pair + 1::4] >= 0) == top)


def test_uniform_noise_range_and_variance():
    u = oracle.uniform_unit(3, 3, 3, 0, N)
    assert np.all(np.abs(u) < math.sqrt(3.0))
    assert abs(u.mean()) <= 5 / math.sqrt(N)
    # Var of a unit-variance uniform sample variance: (9/5 - 1)/N
    assert abs(u.var() - 1.0) <= 5 * math.sqrt(0.8 / N)
    eps = oracle.noise(3, 3, 3, 0, 1000, 0.25, oracle.NOISE_UNIFORM)
    assert np.all(np.abs(eps) <= 0.25 * math.sqrt(3.0))


def test_zero_sigma_draws_nothing():
    assert np.all(oracle.noise(1, 1, 1, 0, 100, 0.0, oracle.NOISE_GAUSSIAN) == 0.0)


def test_offset_consistency():
    # a shard that starts at elem_offset sees the same draws as the whole tensor
    full = oracle.gaussian_z(2, 5, 9, 0, 1000)
    part = oracle.gaussian_z(2, 5, 9, 333, 667)
    np.testing.assert_array_equal(full[333:], part)
    fk = oracle.keep_mask(2, 5, 9, 0, 1000, 0.3)
    pk = oracle.keep_mask(2, 5, 9, 501, 499, 0.3)
    np.testing.assert_array_equal(fk[501:], pk)


def test_laplace_noise_moments_ks_and_range():
    z = oracle.laplace_unit(4, 2, 6, 0, N)
    assert abs(z.mean()) <= 5 / math.sqrt(N)
    # Var of a unit-variance Laplace sample variance: (E z^4 - 1)/N with E z^4 = 6
    assert abs(z.var() - 1.0) <= 5 * math.sqrt(5.0 / N)
    assert stats.kstest(z, "laplace", args=(0.0, 1 / math.sqrt(2))).pvalue > 1e-4
    # the most extreme uniforms give |z| = ln(2^24) / sqrt(2), never infinity
    assert np.all(np.abs(z) <= 24 * math.log(2) / math.sqrt(2) + 1e-12)
    # the median word (u just above 1/2) gives a tiny positive value, its mirror the same negative one
    eps = oracle.noise(4, 2, 6, 0, 1000, 0.5, oracle.NOISE_LAPLACE)
    np.testing.assert_allclose(eps, 0.5 * z[:1000], rtol=1e-15)


def test_laplace_inverse_cdf_special_values():
    # u = (k + 1/2) 2^-24 for k = 2^23 (just above the median) maps to -ln(1 - 2^-24)/sqrt(2) > 0;
    # k = 2^23 - 1 is its mirror image; k = 0 gives the most negative value
    def z_of_k(k):
        u = (k + 0.5) * 2.0 ** -24 - 0.5
        return -math.copysign(1.0, u) * math.log(1 - 2 * abs(u)) / math.sqrt(2)
    assert z_of_k(2 ** 23) == -z_of_k(2 ** 23 - 1) > 0
    assert abs(z_of_k(0) + 24 * math.log(2) / math.sqrt(2)) < 1e-9
    # the oracle uses exactly this map on the top 24 bits of each noise word
    w = oracle.element_words(8, 1, 2, 0, 64, oracle.STREAM_NOISE)
    np.testing.assert_allclose(oracle.laplace_unit(8, 1, 2, 0, 64), [z_of_k(int(x) >> 8) for x in w], rtol=1e-14)
