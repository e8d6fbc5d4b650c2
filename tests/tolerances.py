"""Comparison rules of the GPU path against the oracle, derived from the kernels' fp32 arithmetic.

theta~: the kernel forms t = fl(s/keep) (relative error u = 2^-24 against the oracle's s/keep), then
a = fl(theta0 - t theta0) and b = fl(t theta + a) (the exact-endpoint lerp, two fmas) and
c = fl(sigma z' + b) (z' the hardware Box-Muller value, |z' - z| <= Z_TOL), and rounds c once to the
output type.  With D = theta - theta0 and y the exact value, the three roundings and t's give
|c - y| <= E = u (|t| |D| + |theta0| |1 - t| + 2 |theta0 + t D| + |eps|) + sigma Z_TOL (to first
order; a factor 1 + 8u covers the rest).  The inner fma's term |theta0| |1 - t| is what the
two-fma lerp pays for being exact at t = 0 and t = 1; for t > 5 (rescaled keep below 1/5) it
exceeds 4u |theta0|, so no bound of the form 2^-22 (|theta0| + |t D| + |eps|) holds for every
element.  The output rounding adds half an ulp of the output type.  Where E is below half an ulp of
y (the "strict" elements, all but a few per million on the benchmark lists) this means "within 1
ulp of the oracle's correctly rounded value"; near zero results the absolute bound E governs.

grad: one fma in fp32 with c = fl(lambda * fl(s/keep)): |err| <= 3u (|g_old| + |lambda t g~|),
well inside the 1e-6 relative bar, which is the bound the tests use.
"""
import numpy as np

U = 2.0 ** -24
Z_TOL = 2e-6          # absolute bound on the standard-normal draw
GRAD_RTOL = 1e-6      # relative bound on the fp32 gradient accumulation


def bf16_bits_to_f64(bits):
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def _ulp_bf16(x):
    x = np.abs(np.asarray(x, dtype=np.float64))
    e = np.frexp(x)[1]
    return np.ldexp(1.0, np.maximum(e - 8, -133))


def _ulp_f32(x):
    x = np.abs(np.asarray(x, dtype=np.float64))
    e = np.frexp(x)[1]
    return np.ldexp(1.0, np.maximum(e - 24, -149))


def ordered(bits16):
    """bf16 bit patterns mapped to integers that are monotone in value."""
    b = np.asarray(bits16, dtype=np.int64)
    return np.where(b & 0x8000, 0x8000 - (b & 0x7FFF), 0x8000 + b)


def theta_tilde_bound(theta, theta0, t, eps, sigma):
    """E above: the kernel's fp32 error before the output rounding (fp64 arrays; t = 0 where dropped)."""
    d = theta - theta0
    lin = np.abs(theta0 + t * d)
    return (U * (np.abs(t) * np.abs(d) + np.abs(theta0) * np.abs(1.0 - t) + 2.0 * lin + np.abs(eps)) * (1 + 8 * U)
            + Z_TOL * sigma * (1 + 2 * U))


def check_theta_tilde(gpu, out_dtype, y, theta, theta0, t, eps, sigma):
    """Returns (ok, strict).  gpu: uint16 bits (bf16) or float32 values; y: the oracle's
    unrounded fp64 value; theta, theta0: fp64 inputs; t: fp64 coefficient (0 for dropped
    coordinates); eps: the oracle's noise; sigma: the tensor's noise RMS.
    ok: |gpu - y| <= half an output ulp + E.  strict: elements whose fp32 error bound E is below
    half an output ulp of y; there the GPU value is within 1 ulp of the oracle's rounding of y."""
    theta = np.asarray(theta, dtype=np.float64)
    theta0 = np.asarray(theta0, dtype=np.float64)
    t = np.asarray(t, dtype=np.float64)
    E = theta_tilde_bound(theta, theta0, t, eps, sigma)
    if out_dtype == "bf16":
        g = bf16_bits_to_f64(gpu)
        uy = _ulp_bf16(y)
        half = 0.5 * np.maximum(_ulp_bf16(g), uy)
    else:
        g = np.asarray(gpu, dtype=np.float64)
        uy = _ulp_f32(y)
        half = 0.5 * np.maximum(_ulp_f32(g), uy)
    ok = np.abs(g - y) <= half * (1 + 1e-12) + E
    strict = E < 0.5 * uy
    return ok, strict


# Elements under the absolute clause sit near cancellation (|y| within a few ulps of |theta0| + |eps|
# of zero), at a rate the data set: 2.7e-6 to 3.9e-5 of the elements on the workloads.  The tests
# cap them at 1e-3 of a tensor or list, with an allowance of 8 for small tensors, where the count
# is a Poisson draw: at the cap's own rate, one per 1,000 elements, 9 or more in a 1,000-element
# tensor has probability 1.1e-6, while the data's rate gives a handful only rarely (a 1,042-element
# random case held 2 where 0.08 were expected).
NONSTRICT_MAX_FRACTION = 1e-3
NONSTRICT_SMALL_ALLOWANCE = 8


def nonstrict_within_cap(loose, n):
    """Whether `loose` elements under the absolute clause, out of `n`, stay within the cap above."""
    return loose <= max(NONSTRICT_MAX_FRACTION * n, NONSTRICT_SMALL_ALLOWANCE)


def theta_tilde_report(gpu_bits, want_bits, strict):
    """bf16 outputs against the oracle's rounding: (elements, elements under the absolute clause,
    max ulp distance over all elements, max ulp distance over the strict ones)."""
    d = np.abs(ordered(gpu_bits) - ordered(want_bits))
    return d.size, int(np.count_nonzero(~strict)), int(d.max(initial=0)), int(d[strict].max(initial=0))


def check_grad(gpu, oracle, g_old, incr):
    """gpu/oracle: float32 arrays; g_old: previous values; incr: |lambda t g~| in fp64."""
    scale = np.maximum(np.abs(oracle.astype(np.float64)), np.abs(g_old.astype(np.float64)) + np.abs(incr))
    return np.abs(gpu.astype(np.float64) - oracle.astype(np.float64)) <= GRAD_RTOL * scale


def check_adam(gpu, old, oracle_f64, hp, gmag=None):
    """Fused optimizer step: gpu = (theta, m1, m2) float32 arrays; old = (theta, m1, m2) before the
    step; oracle_f64 = (theta, m1, m2, g) from the oracle in fp64.  Bounds from the kernel's fp32
    sequence (g: <= 5u|g| from t, c = lambda t, the product and grad_scale; m1 = fma(1-b1, g-m1, m1):
    8u(|m1_old| + |g|); m2 is a sum of non-negative terms: 16u m2; theta = fma(-lr/bc1, m1/denom,
    theta (1 - lr wd)): 4u(|theta_old| + |theta|) + 24u (lr/bc1)(|m1_old| + |g|)/denom).
    gmag: magnitude of the gradient's terms (|grad_scale| (|acc| + |lambda t m g~|)); defaults to |g|.
    With an accumulator the kernel's error scales with it rather than with |g|, which may cancel.
    Returns three boolean arrays."""
    th_o, m1_o, m2_o, g = oracle_f64
    ga = np.abs(g) if gmag is None else np.asarray(gmag, dtype=np.float64)
    th0, m10, m20 = (np.asarray(x, dtype=np.float64) for x in old)
    k = int(hp["step"])
    b1, b2 = float(np.float32(hp["beta1"])), float(np.float32(hp["beta2"]))
    step_size = float(np.float32(hp["lr"])) / (1 - b1 ** k)
    denom = np.sqrt(m2_o / (1 - b2 ** k)) + float(np.float32(hp["eps"]))
    tiny = 1e-37
    gt, g1, g2 = (np.asarray(x, dtype=np.float64) for x in gpu)
    ok_m1 = np.abs(g1 - m1_o) <= 8 * U * (np.abs(m10) + ga) + tiny
    ok_m2 = np.abs(g2 - m2_o) <= 16 * U * (m2_o + (1 - b2) * ga * ga) + tiny
    ok_th = np.abs(gt - th_o) <= (4 * U * (np.abs(th0) + np.abs(th_o))
                                  + 24 * U * step_size * (np.abs(m10) + ga) / denom + tiny)
    return ok_th, ok_m1, ok_m2


# Squared gradient norm (smat_grad_norm_multi).  Per element the kernel forms g = fl(c g~) or
# fl(fma(c, g~, acc)) with c = fl(lambda fl(s/keep)): |g' - g| <= 3u m, m = |lambda t g~| + |acc|,
# so |g'^2 - g^2| <= 6u m^2 (first order).  Each thread adds its squares with one fp32 fma chain
# (4 elements for each of its 8 quads, at most 32 terms, 31 for the thread that also takes a
# tensor's 1-3 tail elements), then a 6-level butterfly adds the 64 lanes: a sum of non-negative
# terms through at most 38 roundings, within 38u of the exact total.  The later fp64 additions of
# the per-block partials are negligible.  Hence |sumsq_gpu - sumsq| <= 44u * sum(m^2).
SQNORM_ULPS = 44


def check_sqnorm(gpu, oracle_sumsq, m2_sum):
    """gpu: the kernel's sumsq; oracle_sumsq: exact value (fp64); m2_sum: sum of m^2 as above."""
    return abs(float(gpu) - float(oracle_sumsq)) <= SQNORM_ULPS * U * float(m2_sum) + 1e-300


# N-expert merge (smat_merge): acc starts at theta0 and takes acc = fma(t, x, fma(-t, theta0, acc)) for
# every kept expert coordinate: two roundings per expert, each at most u of the magnitude of the
# running sum or of t theta0.  With A = |theta0| + sum_j |t_j| (|x_j| + |theta0|) (over kept
# coordinates) bounding every partial sum, the fp32 value is within (2N + 1) u A of the exact merge;
# the final rounding adds half an ulp of the output type.  For N = 1 this is the simulate's bound.
def check_merge(gpu, out_dtype, y, A, nexp):
    """Returns (ok, strict) like check_theta_tilde: gpu bf16 bits or fp32 values; y the oracle's fp64
    merge; A the magnitude above (fp64 array); nexp the number of experts that contributed."""
    E = (2 * nexp + 1) * U * np.asarray(A, dtype=np.float64)
    if out_dtype == "bf16":
        g = bf16_bits_to_f64(gpu)
        uy = _ulp_bf16(y)
        half = 0.5 * np.maximum(_ulp_bf16(g), uy)
    else:
        g = np.asarray(gpu, dtype=np.float64)
        uy = _ulp_f32(y)
        half = 0.5 * np.maximum(_ulp_f32(g), uy)
    ok = np.abs(g - y) <= half * (1 + 1e-12) + E
    return ok, E < 0.5 * uy
