"""Pins of the oracle's one-step fp64 -> bfloat16 rounding (nearest, ties to even)."""
import numpy as np
import torch

import oracle


def _bits_of_torch_bf16(x32: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(x32.astype(np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_matches_torch_for_float32_inputs():
    # for values already in float32 a single rounding equals torch's float32 -> bf16 (RNE)
    rng = np.random.default_rng(3)
    vals = [rng.standard_normal(100000).astype(np.float32) * 0.02,
            rng.standard_normal(10000).astype(np.float32) * 1e30,
            (rng.standard_normal(10000) * 1e-39).astype(np.float32),   # float32 subnormals
            np.array([0.0, -0.0, 1.0, -1.0, 3.0e38, -3.0e38, 1e-45, 2 ** -126, 2 ** -133], dtype=np.float32)]
    # exact ties: bf16 value + half a bf16 ulp (low 16 bits = 0x8000)
    ties = (rng.integers(0x0080, 0x7F00, size=5000, dtype=np.uint32) << 16) | np.uint32(0x8000)
    vals.append(ties.view(np.float32))
    for v in vals:
        got = oracle.round_to_bf16_bits(v.astype(np.float64))
        want = _bits_of_torch_bf16(v)
        np.testing.assert_array_equal(got, want)


def _bf16_neighbours(bits: np.ndarray):
    b = bits.astype(np.int64)
    # step one bf16 ulp up/down in magnitude via the integer encoding
    return (b + 1).astype(np.uint16), np.maximum(b - 1, 0).astype(np.uint16)


def test_nearest_with_ties_to_even_for_float64_inputs():
    rng = np.random.default_rng(4)
    x = rng.standard_normal(200000) * 0.03
    x = x[np.abs(x) > 1e-30]
    bits = oracle.round_to_bf16_bits(x)
    v = oracle.bf16_bits_to_f64(bits)
    up, down = _bf16_neighbours(bits & np.uint16(0x7FFF))
    sign = np.where(bits & np.uint16(0x8000), -1.0, 1.0)
    vu = sign * oracle.bf16_bits_to_f64(up)
    vd = sign * oracle.bf16_bits_to_f64(down)
    err = np.abs(v - x)
    assert np.all(err <= np.abs(vu - x))
    assert np.all(err <= np.abs(vd - x))
    # exact midpoints between neighbours go to the even encoding
    lo_bits = (rng.integers(0x3C00, 0x4100, size=2000)).astype(np.uint16)
    lo = oracle.bf16_bits_to_f64(lo_bits)
    hi = oracle.bf16_bits_to_f64((lo_bits.astype(np.int64) + 1).astype(np.uint16))
    mid = 0.5 * (lo + hi)
    got = oracle.round_to_bf16_bits(mid)
    want = np.where(lo_bits % 2 == 0, lo_bits, lo_bits + 1).astype(np.uint16)
    np.testing.assert_array_equal(got, want)
    # one part in 2^40 above a midpoint is no longer a tie: it rounds away from lo
    got = oracle.round_to_bf16_bits(mid * (1 + 2.0 ** -40))
    np.testing.assert_array_equal(got, (lo_bits.astype(np.int64) + 1).astype(np.uint16))


def test_no_double_rounding():
    # a value just above a bf16 midpoint that float32 would round onto the midpoint:
    # rounding fp64 -> f32 -> bf16 would tie to even, the single rounding must go up
    lo_bits = np.array([0x3F80, 0x3F82, 0x4000], dtype=np.uint16)  # even encodings
    lo = oracle.bf16_bits_to_f64(lo_bits)
    hi = oracle.bf16_bits_to_f64(lo_bits + 1)
    x = 0.5 * (lo + hi) + (hi - lo) * 2.0 ** -30
    assert np.all(x.astype(np.float32).astype(np.float64) == 0.5 * (lo + hi))
    np.testing.assert_array_equal(oracle.round_to_bf16_bits(x), lo_bits + 1)


def test_overflow_and_nan():
    big = (2.0 - 2.0 ** -8) * 2.0 ** 127     # midpoint above the largest bf16: rounds to inf
    got = oracle.round_to_bf16_bits(np.array([big, -big, np.inf, np.nan]))
    assert got[0] == 0x7F80 and got[1] == 0xFF80 and got[2] == 0x7F80
    assert (got[3] & 0x7F80) == 0x7F80 and (got[3] & 0x007F) != 0
