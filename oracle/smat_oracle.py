"""CPU oracle for SMAT's per-step parameter transform (test infrastructure only).

This module is a plain, slow, fp64 NumPy statement of what the HIP path
computes.  It exists to check that path: only the tests, the package's smoke
check and the benchmark's CPU-baseline leg may import it.  It shares no code
with the HIP path and imports nothing from it.

What it states (paper: "SMAT: Simple and Efficient Merge-Aware Training"):

* simulated merged state  theta~ = theta0 + alpha * m (.) Delta + eps,
  Delta = theta - theta0, one scalar alpha (called ``s`` here) per tensor
  (Sec. 4.1, Eq. smat-state);
* DARE-style mask: coordinate dropped with probability p = 1 - keep, kept ones
  rescaled by 1/keep (Sec. 4.1, Eq. smat-mask);
* Perturb: zero-mean noise of RMS sigma; the Gaussian form is produced by the
  Box-Muller transform (Sec. 4.1, "Perturb");
* gradient through the simulation: grad_theta += lambda * alpha * m (.) g~,
  zero where the coordinate was dropped (Sec. 4.2, Eq. smat-gradient),
  lambda being the simulated-loss weight (Eq. smat-objective);
* storage switching between expert and simulated storage, and the periodic
  schedule (Sec. 4.3, "Periodic scheduling", "Parameter storage switching";
  App. "Implementation details").

Readings where the paper is silent (it names Triton kernels that sample masks
and noise in-kernel but gives no generator):

* random words: Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw,
  "Parallel random numbers: as easy as 1, 2, 3", SC'11), key = 64-bit seed,
  counter = (g_lo, g_hi, tensor_id, step*4 + stream) where g = e >> 2 for the
  global element index e = elem_offset + i; element e takes word e & 3.
  Stream 0 draws the mask, stream 1 the noise;
* the step's shared scale alpha ~ U[alpha_min, 1], when drawn from the same
  generator: word 0 of counter (0, 0, 0, step*4 + 2) (stream 2, group 0 of
  tensor id 0), u = (w0 >> 8) 2^-24, alpha = alpha_min + (1 - alpha_min) u;
* mask: kept iff word < floor(keep * 2^32); keep >= 1 keeps everything and
  keep <= 0 drops everything without drawing;
* Gaussian noise: lanes (0, 1) of a group pair words (w0, w1), lanes (2, 3)
  pair (w2, w3); u1 = ((a >> 8) + 1) 2^-24 in (0, 1], u2 = (b >> 8) 2^-24 in
  [0, 1); r = sqrt(-2 ln u1); even lane r cos(2 pi u2), odd lane r sin(2 pi u2);
* uniform noise (the paper's default, Sec. 4.1): eps = sigma sqrt(3) (2u - 1)
  with u = ((w >> 8) + 0.5) 2^-24, one word per element;
* Laplace noise at the same RMS (compared in Sec. 4.1): with the same u,
  eps = -sigma sign(u - 1/2) ln(1 - 2|u - 1/2|) / sqrt(2) (inverse CDF of a
  Laplace law of scale sigma / sqrt(2), whose variance is sigma^2);
* all arithmetic in fp64 from the stored input values, one final rounding to
  the output type (round to nearest even).
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence

import numpy as np

# ------------------------------------------------------------------ Philox4x32
# Constants of Philox4x32 (Salmon et al., SC'11, Sec. on the Philox family).
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
MASK32 = 0xFFFFFFFF

STREAM_MASK = 0
STREAM_NOISE = 1
STREAM_SCALE = 2

NOISE_GAUSSIAN = 0
NOISE_UNIFORM = 1
NOISE_LAPLACE = 2

EXPERT = 0
SIMULATED = 1


def philox4x32(c0, c1, c2, c3, k0: int, k1: int, rounds: int = 10):
    """Philox4x32-R bijection on a 128-bit counter under a 64-bit key.

    Each round multiplies words 0 and 2 by the two round constants (full
    64-bit products), swaps the halves into the new state and mixes in the
    key; the key is bumped by the Weyl constants between rounds.  Inputs are
    array-likes of 32-bit values; returns four uint32 arrays.
    """
    c = [np.asarray(x, dtype=np.uint64) & np.uint64(MASK32) for x in (c0, c1, c2, c3)]
    shape = np.broadcast_shapes(*(x.shape for x in c))
    c = [np.broadcast_to(x, shape).copy() for x in c]
    key0, key1 = int(k0) & MASK32, int(k1) & MASK32
    m32 = np.uint64(MASK32)
    for _ in range(rounds):
        p0 = np.uint64(PHILOX_M0) * c[0]
        p1 = np.uint64(PHILOX_M1) * c[2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & m32
        hi1, lo1 = p1 >> np.uint64(32), p1 & m32
        c = [hi1 ^ c[1] ^ np.uint64(key0), lo1, hi0 ^ c[3] ^ np.uint64(key1), lo0]
        key0 = (key0 + PHILOX_W0) & MASK32
        key1 = (key1 + PHILOX_W1) & MASK32
    return tuple(x.astype(np.uint32) for x in c)


def _check_key(seed: int, step: int, tensor_id: int) -> None:
    if not (0 <= seed < 2 ** 64):
        raise ValueError("seed must be a 64-bit unsigned value")
    if not (0 <= step < 2 ** 30):
        raise ValueError("step must be in [0, 2^30)")
    if not (0 <= tensor_id < 2 ** 32):
        raise ValueError("tensor_id must be a 32-bit unsigned value")


def group_words(seed: int, step: int, tensor_id: int, groups, stream: int):
    """The four Philox words of each 4-element group index in `groups`."""
    _check_key(seed, step, tensor_id)
    g = np.asarray(groups, dtype=np.uint64)
    c0 = g & np.uint64(MASK32)
    c1 = g >> np.uint64(32)
    c2 = np.uint64(tensor_id)
    c3 = np.uint64(((step << 2) | stream) & MASK32)
    return philox4x32(c0, c1, c2, c3, seed & MASK32, seed >> 32)


def scale_draw(seed: int, step: int, alpha_min: float) -> float:
    """The scale shared by every coordinate in one simulated update, alpha ~ U[alpha_min, 1]
    (Sec. 4.1, "Scale"), as a function of (seed, step): word 0 of the counter (0, 0, 0, 4 step + 2)
    gives u = (w0 >> 8) 2^-24 in [0, 1); alpha = alpha_min + (1 - alpha_min) u, with alpha_min taken
    as fp32, formed in fp64 and rounded once to fp32 (nearest even)."""
    a = float(np.float32(alpha_min))
    if not (0.0 <= a <= 1.0):
        raise ValueError("alpha_min must lie in [0, 1]")
    w0 = int(group_words(seed, step, 0, [0], STREAM_SCALE)[0][0])
    u = float(w0 >> 8) * 2.0 ** -24
    return float(np.float32(a + (1.0 - a) * u))


def element_words(seed: int, step: int, tensor_id: int, elem_offset: int, n: int, stream: int) -> np.ndarray:
    """One 32-bit word per element: word (e & 3) of group (e >> 2), e = elem_offset + i."""
    e = np.uint64(elem_offset) + np.arange(n, dtype=np.uint64)
    w = group_words(seed, step, tensor_id, e >> np.uint64(2), stream)
    lane = (e & np.uint64(3)).astype(np.int64)
    stacked = np.stack(w)  # (4, n)
    return stacked[lane, np.arange(n)]


# ------------------------------------------------------------------ Mask
def mask_threshold(keep: float) -> Optional[int]:
    """floor(keep * 2^32) for 0 < keep < 1; None when no draw is needed."""
    k = float(np.float32(keep))
    if k >= 1.0 or k <= 0.0:
        return None
    return int(math.floor(k * 2.0 ** 32))


def keep_mask(seed: int, step: int, tensor_id: int, elem_offset: int, n: int, keep: float) -> np.ndarray:
    """Boolean kept-coordinate mask (Eq. smat-mask with p = 1 - keep)."""
    k = float(np.float32(keep))
    if k >= 1.0:
        return np.ones(n, dtype=bool)
    if k <= 0.0:
        return np.zeros(n, dtype=bool)
    thr = mask_threshold(k)
    w = element_words(seed, step, tensor_id, elem_offset, n, STREAM_MASK).astype(np.uint64)
    return w < np.uint64(thr)


def mask_values(kept: np.ndarray, keep: float, rescale: bool) -> np.ndarray:
    """m_k in fp64: 0 for dropped coordinates, 1/keep (or 1 without rescale) for kept ones."""
    k = float(np.float32(keep))
    if k <= 0.0:
        return np.zeros(kept.shape, dtype=np.float64)
    val = (1.0 / k) if (rescale and k < 1.0) else 1.0
    return np.where(kept, val, 0.0)


# ------------------------------------------------------------------ Noise
def box_muller(a_words, b_words):
    """Gaussian pair from two words: (r cos 2 pi u2, r sin 2 pi u2), fp64."""
    a = np.asarray(a_words, dtype=np.uint64)
    b = np.asarray(b_words, dtype=np.uint64)
    u1 = ((a >> np.uint64(8)).astype(np.float64) + 1.0) * 2.0 ** -24
    u2 = (b >> np.uint64(8)).astype(np.float64) * 2.0 ** -24
    r = np.sqrt(-2.0 * np.log(u1))
    return r * np.cos(2.0 * np.pi * u2), r * np.sin(2.0 * np.pi * u2)


def gaussian_z(seed: int, step: int, tensor_id: int, elem_offset: int, n: int) -> np.ndarray:
    """Standard-normal draw per element from the noise stream (fp64)."""
    e = np.uint64(elem_offset) + np.arange(n, dtype=np.uint64)
    w0, w1, w2, w3 = group_words(seed, step, tensor_id, e >> np.uint64(2), STREAM_NOISE)
    zc01, zs01 = box_muller(w0, w1)
    zc23, zs23 = box_muller(w2, w3)
    lane = (e & np.uint64(3)).astype(np.int64)
    return np.choose(lane, [zc01, zs01, zc23, zs23])


def uniform_unit(seed: int, step: int, tensor_id: int, elem_offset: int, n: int) -> np.ndarray:
    """Zero-mean, unit-variance uniform draw per element: sqrt(3) (2u - 1)."""
    w = element_words(seed, step, tensor_id, elem_offset, n, STREAM_NOISE).astype(np.uint64)
    u = ((w >> np.uint64(8)).astype(np.float64) + 0.5) * 2.0 ** -24
    return math.sqrt(3.0) * (2.0 * u - 1.0)


def laplace_unit(seed: int, step: int, tensor_id: int, elem_offset: int, n: int) -> np.ndarray:
    """Zero-mean, unit-variance Laplace draw per element by inversion of its CDF."""
    w = element_words(seed, step, tensor_id, elem_offset, n, STREAM_NOISE).astype(np.uint64)
    u = ((w >> np.uint64(8)).astype(np.float64) + 0.5) * 2.0 ** -24 - 0.5   # in (-1/2, 1/2), never 0
    return -np.sign(u) * np.log(1.0 - 2.0 * np.abs(u)) / math.sqrt(2.0)


def noise(seed: int, step: int, tensor_id: int, elem_offset: int, n: int, sigma: float, kind: int) -> np.ndarray:
    """eps in fp64 (Sec. 4.1, "Perturb"); sigma == 0 gives exact zeros without drawing."""
    sg = float(np.float32(sigma))
    if sg == 0.0:
        return np.zeros(n, dtype=np.float64)
    if kind == NOISE_GAUSSIAN:
        return sg * gaussian_z(seed, step, tensor_id, elem_offset, n)
    if kind == NOISE_UNIFORM:
        return sg * uniform_unit(seed, step, tensor_id, elem_offset, n)
    if kind == NOISE_LAPLACE:
        return sg * laplace_unit(seed, step, tensor_id, elem_offset, n)
    raise ValueError(f"unknown noise kind {kind}")


# ------------------------------------------------------------------ rounding
def round_to_bf16_bits(x) -> np.ndarray:
    """Round fp64 values to bfloat16 (nearest, ties to even) in one step; uint16 bits."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.float64)
    finite = np.isfinite(x)
    xf = np.where(finite, x, 0.0)
    mant, expo = np.frexp(np.abs(xf))           # |x| = mant * 2^expo, mant in [0.5, 1)
    # bf16 keeps 8 significant bits; below 2^-126 the spacing is fixed at 2^-133
    ulp_exp = np.maximum(expo - 8, -133)
    scaled = np.ldexp(np.abs(xf), -ulp_exp)
    rounded = np.ldexp(np.rint(scaled), ulp_exp)  # np.rint rounds half to even
    rounded = np.copysign(rounded, xf)
    bf16_max = (2.0 - 2.0 ** -7) * 2.0 ** 127
    rounded = np.where(np.abs(rounded) > bf16_max, np.copysign(np.inf, rounded), rounded)
    out[:] = np.where(finite, rounded, x)
    f32 = out.astype(np.float32)
    bits = (f32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    bits = np.where(nan, np.uint16(0x7FC0), bits)
    return bits


def bf16_bits_to_f64(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def round_to(x, dtype: str) -> np.ndarray:
    """Round fp64 to the storage dtype: "bf16" -> uint16 bits, "f32" -> float32."""
    if dtype == "bf16":
        return round_to_bf16_bits(x)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float64).astype(np.float32)
    raise ValueError(dtype)


def as_f64(values, dtype: str) -> np.ndarray:
    """Stored values (bf16 bits as uint16, or float32/float64) as fp64."""
    if dtype == "bf16":
        return bf16_bits_to_f64(values)
    return np.asarray(values).astype(np.float64)


# ------------------------------------------------------------------ parameters
def validate_params(s: float, keep: float, sigma: float, rescale: int = 1, noise_kind: int = 0) -> None:
    """Argument rules of the operations: keep in [0, 1], sigma finite and >= 0, s finite."""
    if not math.isfinite(s):
        raise ValueError("scale must be finite")
    if not (math.isfinite(keep) and 0.0 <= keep <= 1.0):
        raise ValueError("keep must lie in [0, 1]")
    if not (math.isfinite(sigma) and sigma >= 0.0):
        raise ValueError("sigma must be finite and non-negative")
    if noise_kind not in (NOISE_GAUSSIAN, NOISE_UNIFORM, NOISE_LAPLACE):
        raise ValueError("unknown noise kind")


def coefficient(s: float, keep: float, rescale: int) -> float:
    """alpha * m for a kept coordinate, exact in fp64: s / keep with rescale, else s."""
    k = float(np.float32(keep))
    sv = float(np.float32(s))
    if rescale and 0.0 < k < 1.0:
        return sv / k
    return sv


# ------------------------------------------------------------------ operations
def simulate_f64(theta, theta0, theta0_dtype: str, p: dict, seed: int, step: int, tensor_id: int,
                 elem_offset: int = 0):
    """Unrounded theta~ in fp64 plus the kept mask and the noise (Eq. smat-state).

    theta: float array (its values are used exactly); theta0: stored values
    (uint16 bf16 bits for "bf16", else a float array).  Returns (y, kept, eps).
    """
    validate_params(p["s"], p["keep"], p["sigma"], p.get("rescale", 1), p.get("noise_kind", 0))
    th = np.asarray(theta).astype(np.float64).ravel()
    t0 = as_f64(np.asarray(theta0).ravel(), theta0_dtype)
    n = th.size
    if t0.size != n:
        raise ValueError("theta and theta0 differ in size")
    kept = keep_mask(seed, step, tensor_id, elem_offset, n, p["keep"])
    m = mask_values(kept, p["keep"], p.get("rescale", 1))
    alpha = float(np.float32(p["s"]))
    eps = noise(seed, step, tensor_id, elem_offset, n, p["sigma"], p.get("noise_kind", 0))
    y = t0 + alpha * m * (th - t0) + eps
    return y, kept, eps


def simulate(theta, theta0, theta0_dtype: str, out_dtype: str, p: dict, seed: int, step: int,
             tensor_id: int, elem_offset: int = 0) -> np.ndarray:
    """theta~ rounded once to `out_dtype` (uint16 bits for bf16, float32 for f32)."""
    y, _, _ = simulate_f64(theta, theta0, theta0_dtype, p, seed, step, tensor_id, elem_offset)
    return round_to(y, out_dtype)


def backward_accum(grad_sim, grad_sim_dtype: str, grad_theta, p: dict, lam: float, seed: int, step: int,
                   tensor_id: int, elem_offset: int = 0) -> np.ndarray:
    """grad_theta + lambda * alpha * m (.) g~ (Eq. smat-gradient, weighted by lambda).

    Dropped coordinates keep their previous fp32 value bit for bit; kept ones
    get the fp64 sum rounded once to fp32.
    """
    validate_params(p["s"], p["keep"], p["sigma"], p.get("rescale", 1), p.get("noise_kind", 0))
    if not math.isfinite(lam):
        raise ValueError("lambda must be finite")
    g = as_f64(np.asarray(grad_sim).ravel(), grad_sim_dtype)
    gt = np.asarray(grad_theta, dtype=np.float32).ravel()
    n = gt.size
    if g.size != n:
        raise ValueError("grad_sim and grad_theta differ in size")
    kept = keep_mask(seed, step, tensor_id, elem_offset, n, p["keep"])
    m = mask_values(kept, p["keep"], p.get("rescale", 1))
    lam32 = float(np.float32(lam))
    alpha = float(np.float32(p["s"]))
    new = (gt.astype(np.float64) + lam32 * alpha * m * g).astype(np.float32)
    return np.where(kept, new, gt)


# ------------------------------------------------------------------ fused optimizer step
def validate_adamw(hp: dict) -> None:
    for k in ("lr", "beta1", "beta2", "eps", "weight_decay", "grad_scale"):
        if not math.isfinite(hp[k]):
            raise ValueError(f"{k} must be finite")
    if not (0.0 <= hp["beta1"] < 1.0 and 0.0 <= hp["beta2"] < 1.0):
        raise ValueError("betas must lie in [0, 1)")
    if hp["eps"] <= 0.0 or hp["lr"] < 0.0 or hp["weight_decay"] < 0.0:
        raise ValueError("eps must be > 0, lr and weight_decay >= 0")
    if int(hp["step"]) < 1:
        raise ValueError("step must be >= 1")


def adamw_update(theta, exp_avg, exp_avg_sq, grad, hp: dict):
    """One decoupled-weight-decay Adam step (Loshchilov & Hutter; Adam when weight_decay = 0) in fp64:
    m1 = b1 m1 + (1 - b1) g, m2 = b2 m2 + (1 - b2) g^2,
    theta = theta (1 - lr wd) - lr (m1 / (1 - b1^k)) / (sqrt(m2 / (1 - b2^k)) + eps).
    Inputs are arrays (any float dtype, used exactly); returns the fp64 results."""
    validate_adamw(hp)
    f = lambda x: float(np.float32(x))
    lr, b1, b2, eps, wd = f(hp["lr"]), f(hp["beta1"]), f(hp["beta2"]), f(hp["eps"]), f(hp["weight_decay"])
    k = int(hp["step"])
    th = np.asarray(theta).astype(np.float64)
    m1 = b1 * np.asarray(exp_avg).astype(np.float64) + (1.0 - b1) * grad
    m2 = b2 * np.asarray(exp_avg_sq).astype(np.float64) + (1.0 - b2) * grad * grad
    bc1 = 1.0 - b1 ** k
    bc2 = 1.0 - b2 ** k
    new = th * (1.0 - lr * wd) - lr * (m1 / bc1) / (np.sqrt(m2 / bc2) + eps)
    return new, m1, m2


def simulated_gradient(grad_sim, grad_sim_dtype: str, p: dict, lam: float, seed: int, step: int, tensor_id: int,
                       elem_offset: int = 0, grad_acc=None, grad_scale: float = 1.0) -> np.ndarray:
    """grad_scale * (grad_acc + lambda * alpha * m (.) g~) in fp64 (Eq. smat-gradient, weighted by lambda)."""
    validate_params(p["s"], p["keep"], p["sigma"], p.get("rescale", 1), p.get("noise_kind", 0))
    g = as_f64(np.asarray(grad_sim).ravel(), grad_sim_dtype)
    kept = keep_mask(seed, step, tensor_id, elem_offset, g.size, p["keep"])
    m = mask_values(kept, p["keep"], p.get("rescale", 1))
    out = float(np.float32(lam)) * float(np.float32(p["s"])) * m * g
    if grad_acc is not None:
        out = out + np.asarray(grad_acc).astype(np.float64).ravel()
    return float(np.float32(grad_scale)) * out


def adamw_fused(grad_sim, grad_sim_dtype: str, theta, exp_avg, exp_avg_sq, p: dict, lam: float, hp: dict,
                seed: int, step: int, tensor_id: int, elem_offset: int = 0, grad_acc=None):
    """The optimizer update of a simulated step fed directly by the simulated-loss gradient; the
    expert storage and its optimizer state are updated (App. "Training and Scheduling Details",
    "Implementation details": the optimizer runs on the restored storage, weight decay included).
    Returns (theta, exp_avg, exp_avg_sq) as float32 arrays and the fp64 values before rounding."""
    g = simulated_gradient(grad_sim, grad_sim_dtype, p, lam, seed, step, tensor_id, elem_offset, grad_acc,
                           hp["grad_scale"])
    th, m1, m2 = adamw_update(np.asarray(theta).ravel(), np.asarray(exp_avg).ravel(),
                              np.asarray(exp_avg_sq).ravel(), g, hp)
    return (th.astype(np.float32), m1.astype(np.float32), m2.astype(np.float32)), (th, m1, m2, g)


def grad_sqnorm(grad_sim, grad_sim_dtype: str, p: dict, lam: float, seed: int, step: int, tensor_id: int,
                elem_offset: int = 0, grad_acc=None) -> float:
    """Squared L2 norm of the expert gradient [grad_acc +] lambda * alpha * m (.) g~ of one tensor,
    in fp64 (the quantity gradient-norm clipping measures before the optimizer step)."""
    g = simulated_gradient(grad_sim, grad_sim_dtype, p, lam, seed, step, tensor_id, elem_offset, grad_acc)
    return float(np.dot(g, g))


def clip_coefficient(total_norm: float, max_norm: float) -> float:
    """Norm clipping with the rule of torch.nn.utils.clip_grad_norm_ (L2 norm): the gradient is
    multiplied by min(1, max_norm / (total_norm + 1e-6))."""
    if not (math.isfinite(max_norm) and max_norm > 0.0):
        raise ValueError("max_norm must be finite and > 0")
    return min(1.0, max_norm / (total_norm + 1e-6))


# ------------------------------------------------------------------ ragged lists
def grad_sqnorm_multi(grad_sims: Sequence, grad_sim_dtype: str, params: Sequence[dict], lam: float, seed: int,
                      step: int, tensor_ids: Sequence[int], elem_offsets: Optional[Sequence[int]] = None,
                      grad_accs: Optional[Sequence] = None) -> float:
    """Squared L2 norm of the expert gradient over a list of tensors (or shards of tensors), in fp64."""
    offs = elem_offsets if elem_offsets is not None else [0] * len(grad_sims)
    total = 0.0
    for i in range(len(grad_sims)):
        total += grad_sqnorm(grad_sims[i], grad_sim_dtype, params[i], lam, seed, step, tensor_ids[i], offs[i],
                             None if grad_accs is None else grad_accs[i])
    return total


def simulate_multi(thetas: Sequence, theta0s: Sequence, theta0_dtype: str, out_dtype: str,
                   params: Sequence[dict], seed: int, step: int, tensor_ids: Sequence[int],
                   elem_offsets: Optional[Sequence[int]] = None) -> List[np.ndarray]:
    if len(set(tensor_ids)) != len(tensor_ids):
        raise ValueError("duplicate tensor ids")
    offs = elem_offsets if elem_offsets is not None else [0] * len(thetas)
    return [simulate(thetas[i], theta0s[i], theta0_dtype, out_dtype, params[i], seed, step,
                     tensor_ids[i], offs[i]) for i in range(len(thetas))]


def backward_accum_multi(grad_sims: Sequence, grad_sim_dtype: str, grad_thetas: Sequence,
                         params: Sequence[dict], lam: float, seed: int, step: int,
                         tensor_ids: Sequence[int], elem_offsets: Optional[Sequence[int]] = None
                         ) -> List[np.ndarray]:
    if len(set(tensor_ids)) != len(tensor_ids):
        raise ValueError("duplicate tensor ids")
    offs = elem_offsets if elem_offsets is not None else [0] * len(grad_sims)
    return [backward_accum(grad_sims[i], grad_sim_dtype, grad_thetas[i], params[i], lam, seed, step,
                           tensor_ids[i], offs[i]) for i in range(len(grad_sims))]


# ------------------------------------------------------------------ merging (evaluation side)
def validate_merge_term(t: dict) -> None:
    g, k = float(t["gamma"]), float(t["keep"])
    if not math.isfinite(g):
        raise ValueError("gamma must be finite")
    if not (0.0 <= k <= 1.0):
        raise ValueError("keep must lie in [0, 1]")
    _check_key(int(t["seed"]), int(t["step"]), 0)


def merge_f64(experts: Sequence, expert_dtype: str, theta0, theta0_dtype: str, terms: Sequence[dict],
              tensor_id: int, elem_offset: int = 0) -> np.ndarray:
    """Merged parameters in fp64 (Eq. merged-state):
        theta_merge = theta0 + sum_j alpha_j m_j (.) (theta_j - theta0)
    with a scalar weight alpha_j = gamma_j per expert (Task Arithmetic: all gamma_j = gamma; weight
    averaging: gamma_j = 1/N) and DARE masks m_j (coordinate dropped with probability 1 - keep_j,
    kept ones rescaled by 1/keep_j unless rescale is 0; keep_j = 1 leaves the task vector whole).
    Expert j's mask is drawn like a training mask, from its own (seed, step) and the tensor's id and
    element offsets, so one expert with (gamma = s, keep, seed, step) gives the simulated state of
    that step without noise.  terms: one dict(gamma, keep, rescale=1, seed, step) per expert."""
    if len(experts) != len(terms):
        raise ValueError("one term per expert")
    y = as_f64(np.asarray(theta0).ravel(), theta0_dtype)
    t0 = y.copy()
    n = t0.size
    for x, t in zip(experts, terms):
        validate_merge_term(t)
        th = as_f64(np.asarray(x).ravel(), expert_dtype)
        if th.size != n:
            raise ValueError("an expert differs in size from theta0")
        kept = keep_mask(int(t["seed"]), int(t["step"]), tensor_id, elem_offset, n, t["keep"])
        m = mask_values(kept, t["keep"], t.get("rescale", 1))
        y = y + float(np.float32(t["gamma"])) * m * (th - t0)
    return y


def merge(experts: Sequence, expert_dtype: str, theta0, theta0_dtype: str, out_dtype: str, terms: Sequence[dict],
          tensor_id: int, elem_offset: int = 0) -> np.ndarray:
    """merge_f64 rounded once to out_dtype (uint16 bits for bf16, float32 for f32)."""
    return round_to(merge_f64(experts, expert_dtype, theta0, theta0_dtype, terms, tensor_id, elem_offset), out_dtype)


# ------------------------------------------------------------------ schedule + switch
def is_simulated_step(step: int, period: int = 4) -> bool:
    """Periodic scheduling: t-1 ordinary steps then one simulated step (Sec. 4.3).

    Reading: the simulated step closes each cycle, i.e. step mod t == t - 1
    (0-based), so ordinary steps come first.
    """
    if period < 1:
        raise ValueError("period must be >= 1")
    return step % period == period - 1


class StateError(RuntimeError):
    pass


class StorageSwitch:
    """Expert / simulated storage state machine (Sec. 4.3 and App. "Implementation details").

    The model reads its weights through an active view.  EXPERT shows the
    expert (fp32 master) storage, SIMULATED shows the reusable buffer that
    holds theta~.  The optimizer only ever sees EXPERT.  In offload mode the
    frozen base lives in host memory and is copied into the buffer when the
    state returns to EXPERT, so the buffer holds theta0 before the next
    simulate.
    """

    def __init__(self, theta: Sequence, theta0: Sequence, offload: bool = False):
        self.theta = [np.array(x, copy=True) for x in theta]
        self.theta0 = [np.array(x, copy=True) for x in theta0]
        self.offload = offload
        self.state = EXPERT
        self.fresh = False      # buffer holds theta~ of the latest simulate
        # resident mode: buffer starts empty; offload mode: buffer starts as theta0
        self.buffer = [np.array(x, copy=True) for x in theta0] if offload else [None] * len(theta0)

    def simulate(self, out: Sequence) -> None:
        if self.state != EXPERT:
            raise StateError("simulate while the simulated storage is active")
        if self.offload and self.fresh:
            # the buffer is the device's only copy of the base in offload mode and the simulate
            # writes theta~ over it: the base is back only after the next restore
            raise StateError("offload mode: the buffer holds theta~ until the next restore refills theta0")
        self.buffer = [np.array(x, copy=True) for x in out]
        self.fresh = True

    def switch(self, to: int) -> None:
        if to == SIMULATED:
            if self.state == SIMULATED:
                raise StateError("already simulated")
            if not self.fresh:
                raise StateError("no simulated weights since the last restore")
            self.state = SIMULATED
        elif to == EXPERT:
            if self.state == EXPERT:
                return  # restoring the expert view is idempotent
            self.state = EXPERT
            self.fresh = False
            if self.offload:
                self.buffer = [np.array(x, copy=True) for x in self.theta0]
        else:
            raise ValueError("unknown storage state")

    def active(self) -> list:
        return self.buffer if self.state == SIMULATED else self.theta
