"""GPU parity of the single-tensor entry points (smat_simulate, smat_backward_accum,
smat_debug_draws) against the CPU oracle, through the C ABI."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_33437_amd as smat
import workloads
from helpers import host
from tolerances import Z_TOL, check_grad, check_theta_tilde, nonstrict_within_cap, ordered, theta_tilde_report

pytestmark = pytest.mark.gpu
DEV = "cuda"


def run_simulate(theta, theta0, out, p, seed, step, tid, off=0):
    smat.smat_simulate(theta, theta0, out, p, seed, step, tid, off)
    torch.cuda.synchronize()


def compare_simulate(theta, theta0, out, p, seed, step, tid, off=0):
    """Run the kernel and check every element against the oracle; returns the ulp distances."""
    run_simulate(theta, theta0, out, p, seed, step, tid, off)
    th, _ = host(theta)
    t0, t0_dt = host(theta0)
    got, out_dt = host(out)
    y, kept, eps = oracle.simulate_f64(th, t0, t0_dt, p, seed, step, tid, off)
    coef = np.where(kept, oracle.coefficient(p["s"], p["keep"], p.get("rescale", 1)), 0.0)
    ok, strict = check_theta_tilde(got, out_dt, y, th, oracle.as_f64(t0, t0_dt), coef, eps, p["sigma"])
    bad = np.flatnonzero(~ok)
    assert bad.size == 0, f"{bad.size} mismatches, first at {bad[:5]}: gpu={got[bad[:5]]} y={y[bad[:5]]}"
    if out_dt == "bf16":
        want = oracle.round_to_bf16_bits(y)
        n, loose, worst, worst_strict = theta_tilde_report(got, want, strict)
        print(f"theta~ {n} elements: {loose} under the absolute clause, max {worst} ulp (strict {worst_strict})")
        assert nonstrict_within_cap(loose, n), (loose, n)
        return np.abs(ordered(got) - ordered(want))[strict]
    return None


KEYS = [(0, 0, 0, 0), (0x5EED0003, 17, 41, 4 * 1000 + 3), (2 ** 64 - 1, 2 ** 30 - 1, 2 ** 32 - 1, 2 ** 40 + 1),
        (123456789, 5, 7, 1)]


@pytest.mark.parametrize("seed,step,tid,off", KEYS)
def test_debug_draws_bit_exact(seed, step, tid, off):
    n = 4099
    mw = torch.empty(n, dtype=torch.int32, device=DEV)
    nw = torch.empty(n, dtype=torch.int32, device=DEV)
    kept = torch.empty(n, dtype=torch.uint8, device=DEV)
    z = torch.empty(n, dtype=torch.float32, device=DEV)
    p = dict(s=1.0, keep=0.3, sigma=1.0)
    smat.smat_debug_draws(n, p, seed, step, tid, off, mw, nw, kept, z)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(mw.cpu().numpy().view(np.uint32),
                                  oracle.element_words(seed, step, tid, off, n, oracle.STREAM_MASK))
    np.testing.assert_array_equal(nw.cpu().numpy().view(np.uint32),
                                  oracle.element_words(seed, step, tid, off, n, oracle.STREAM_NOISE))
    np.testing.assert_array_equal(kept.cpu().numpy().astype(bool), oracle.keep_mask(seed, step, tid, off, n, 0.3))
    zo = oracle.gaussian_z(seed, step, tid, off, n)
    assert np.max(np.abs(z.cpu().numpy().astype(np.float64) - zo)) <= Z_TOL


def test_gaussian_z_accuracy_many_draws():
    n = 1 << 22
    z = torch.empty(n, dtype=torch.float32, device=DEV)
    smat.smat_debug_draws(n, dict(s=1.0, keep=1.0, sigma=1.0), 99, 3, 5, 0, z=z)
    torch.cuda.synchronize()
    zo = oracle.gaussian_z(99, 3, 5, 0, n)
    err = np.abs(z.cpu().numpy().astype(np.float64) - zo)
    print(f"max |z_gpu - z| over {n} draws: {err.max():.3e}")
    assert err.max() <= Z_TOL


def test_debug_kept_degenerate_keeps():
    n = 1000
    kept = torch.empty(n, dtype=torch.uint8, device=DEV)
    for keep, want in ((1.0, 1), (0.0, 0)):
        smat.smat_debug_draws(n, dict(s=1.0, keep=keep, sigma=0.0), 1, 2, 3, 0, kept=kept)
        torch.cuda.synchronize()
        assert bool((kept == want).all())


def _c1():
    cfg = workloads.config("c1")
    inp = workloads.make_inputs(cfg, device="cpu")
    return cfg, inp.theta[0].to(DEV), inp.theta0[0].to(DEV), inp.grad_sim[0].to(DEV), inp.grad_theta[0].to(DEV)


@pytest.mark.parametrize("out_dtype", [torch.bfloat16, torch.float32])
def test_simulate_c1(out_dtype):
    cfg, theta, theta0, _, _ = _c1()
    p = dict(s=0.7, keep=0.5, sigma=1e-3, rescale=1, noise_kind=0)
    out = torch.empty(theta.numel(), dtype=out_dtype, device=DEV)
    dist = compare_simulate(theta, theta0, out, p, cfg.smat_seed, 0, 0)
    if dist is not None:
        print(f"bf16 ulp distance histogram: {np.bincount(dist)}")
        assert dist.max(initial=0) <= 1


def test_backward_c1():
    cfg, _, _, gs, gt = _c1()
    gt = gt + torch.randn(gt.shape, device=DEV, generator=torch.Generator(DEV).manual_seed(1)) * 1e-3
    p = dict(s=0.7, keep=0.5, sigma=1e-3, rescale=1, noise_kind=0)
    g_old, _ = host(gt)
    gsn, gs_dt = host(gs)
    smat.smat_backward_accum(gs, gt, p, 1.0, cfg.smat_seed, 0, 0)
    torch.cuda.synchronize()
    got, _ = host(gt)
    want = oracle.backward_accum(gsn, gs_dt, g_old, p, 1.0, cfg.smat_seed, 0, 0)
    kept = oracle.keep_mask(cfg.smat_seed, 0, 0, 0, gt.numel(), 0.5)
    np.testing.assert_array_equal(got.view(np.uint32)[~kept], g_old.view(np.uint32)[~kept])
    incr = np.abs(0.7 / 0.5 * oracle.as_f64(gsn, gs_dt))
    assert check_grad(got, want, g_old, incr).all()


def test_forward_and_backward_masks_agree():
    # coordinates that the backward leaves untouched are exactly those the forward dropped
    n = 1 << 16
    g = torch.Generator(DEV).manual_seed(3)
    theta = torch.randn(n, device=DEV, generator=g) * 0.02
    theta0 = torch.zeros(n, device=DEV, dtype=torch.float32)
    out = torch.empty(n, device=DEV, dtype=torch.float32)
    p = dict(s=1.0, keep=0.37, sigma=0.0)
    smat.smat_simulate(theta, theta0, out, p, 11, 2, 4)
    gt = torch.zeros(n, device=DEV)
    smat.smat_backward_accum(torch.ones(n, device=DEV), gt, p, 1.0, 11, 2, 4)
    torch.cuda.synchronize()
    assert torch.equal(out != 0, gt != 0)


def test_closed_forms_exact():
    n = 100003
    g = torch.Generator(DEV).manual_seed(5)
    theta = torch.randn(n, device=DEV, generator=g) * 0.02 + 0.001
    theta0 = (torch.randn(n, device=DEV, generator=g) * 0.02 + 0.001).to(torch.bfloat16)
    out32 = torch.empty(n, device=DEV, dtype=torch.float32)
    out16 = torch.empty(n, device=DEV, dtype=torch.bfloat16)
    ident = dict(s=1.0, keep=1.0, sigma=0.0)
    smat.smat_simulate(theta, theta0, out32, ident, 1, 1, 1)
    smat.smat_simulate(theta, theta0, out16, ident, 1, 1, 1)
    torch.cuda.synchronize()
    assert torch.equal(out32, theta)
    assert torch.equal(out16.view(torch.int16), theta.to(torch.bfloat16).view(torch.int16))
    for p in (dict(s=0.8, keep=0.0, sigma=0.0), dict(s=0.0, keep=0.4, sigma=0.0)):
        smat.smat_simulate(theta, theta0, out16, p, 1, 1, 1)
        torch.cuda.synchronize()
        assert torch.equal(out16.view(torch.int16), theta0.view(torch.int16))
    # keep = 0 with noise: independent of theta
    p = dict(s=0.8, keep=0.0, sigma=1e-3)
    smat.smat_simulate(theta, theta0, out16, p, 1, 1, 1)
    other = torch.empty_like(out16)
    smat.smat_simulate(theta * 7 + 1, theta0, other, p, 1, 1, 1)
    torch.cuda.synchronize()
    assert torch.equal(out16.view(torch.int16), other.view(torch.int16))
    # backward: s = keep = lambda = 1 is the textbook add
    gt = torch.randn(n, device=DEV, generator=g) * 1e-3
    gs = torch.randn(n, device=DEV, generator=g) * 1e-2
    want = gt + gs
    smat.smat_backward_accum(gs, gt, ident, 1.0, 1, 1, 1)
    torch.cuda.synchronize()
    assert torch.equal(gt, want)


# sizes around quads and chunks; element offsets and base misalignment that force the per-element path;
# offsets whose tiles cross a multiple of 2^34 elements, where the high counter word of the groups changes
@pytest.mark.parametrize("n,shift,off", [(1, 0, 0), (3, 0, 0), (4, 0, 0), (5, 0, 0), (4095, 0, 0),
                                          (16384, 0, 0), (16384 + 7, 0, 0), (3 * 16384 + 1, 0, 4),
                                          (50000, 1, 0), (50000, 0, 2), (50001, 3, 5), (70000, 2, 2 ** 33 + 1),
                                          (70000, 0, 2 ** 34 + 4096), (5000, 0, 2 ** 34 - 1000),
                                          (70001, 0, 2 ** 35 - 30000)])
@pytest.mark.parametrize("dts", [("bf16", "bf16", "bf16"), ("f32", "f32", "f32"), ("f32", "bf16", "bf16")])
def test_ragged_and_misaligned(n, shift, off, dts):
    tmap = {"bf16": torch.bfloat16, "f32": torch.float32}
    t0_dt, out_dt, g_dt = dts
    g = torch.Generator(DEV).manual_seed(n + shift)
    theta = (torch.randn(n + 8, device=DEV, generator=g) * 0.02)[shift:shift + n]
    theta0 = (torch.randn(n + 8, device=DEV, generator=g) * 0.02).to(tmap[t0_dt])[shift:shift + n]
    out = torch.empty(n + 8, device=DEV, dtype=tmap[out_dt])[shift:shift + n]
    p = dict(s=0.55, keep=0.3, sigma=2e-3, rescale=1, noise_kind=0)
    dist = compare_simulate(theta, theta0, out, p, 77, 9, 13, off)
    if dist is not None:
        assert dist.max(initial=0) <= 1
    gs = (torch.randn(n + 8, device=DEV, generator=g) * 1e-2).to(tmap[g_dt])[shift:shift + n]
    gt = (torch.randn(n + 8, device=DEV, generator=g) * 1e-3)[shift:shift + n]
    g_old, _ = host(gt)
    gsn, gs_dt = host(gs)
    smat.smat_backward_accum(gs, gt, p, 0.5, 77, 9, 13, off)
    torch.cuda.synchronize()
    got, _ = host(gt)
    want = oracle.backward_accum(gsn, gs_dt, g_old, p, 0.5, 77, 9, 13, off)
    assert check_grad(got, want, g_old, np.abs(0.5 * 0.55 / 0.3 * oracle.as_f64(gsn, gs_dt))).all()
    kept = oracle.keep_mask(77, 9, 13, off, n, 0.3)
    np.testing.assert_array_equal(got.view(np.uint32)[~kept], g_old.view(np.uint32)[~kept])


def test_uniform_noise_parity_and_range():
    n = 200000
    g = torch.Generator(DEV).manual_seed(8)
    theta = torch.randn(n, device=DEV, generator=g) * 0.02
    theta0 = theta.to(torch.bfloat16)
    out = torch.empty(n, device=DEV, dtype=torch.float32)
    p = dict(s=0.9, keep=0.6, sigma=1e-3, rescale=1, noise_kind=oracle.NOISE_UNIFORM)
    compare_simulate(theta, theta0, out, p, 5, 6, 7)
    # keep = 0 and theta0 exactly representable: theta~ - theta0 = eps stays inside +-sqrt(3) sigma
    p0 = dict(s=0.9, keep=0.0, sigma=1e-3, rescale=1, noise_kind=oracle.NOISE_UNIFORM)
    smat.smat_simulate(theta, theta0, out, p0, 5, 6, 7)
    torch.cuda.synchronize()
    d = (out.double() - theta0.double()).cpu().numpy()
    assert np.all(np.abs(d) <= math.sqrt(3) * 1e-3 + 1e-8)   # + fp32 rounding of theta0 + eps
    assert abs(d.var() - 1e-6) <= 5 * math.sqrt(0.8 / n) * 1e-6


def test_in_place_over_theta0_and_determinism():
    n = 123457
    g = torch.Generator(DEV).manual_seed(9)
    theta = torch.randn(n, device=DEV, generator=g) * 0.02
    base = (torch.randn(n, device=DEV, generator=g) * 0.02).to(torch.bfloat16)
    p = dict(s=0.5, keep=0.25, sigma=1e-3)
    ref = torch.empty_like(base)
    smat.smat_simulate(theta, base, ref, p, 3, 4, 5)
    again = torch.empty_like(base)
    smat.smat_simulate(theta, base, again, p, 3, 4, 5)
    buf = base.clone()
    smat.smat_simulate(theta, buf, buf, p, 3, 4, 5)       # out aliases theta0
    torch.cuda.synchronize()
    assert torch.equal(ref.view(torch.int16), again.view(torch.int16))
    assert torch.equal(ref.view(torch.int16), buf.view(torch.int16))


def test_errors_through_the_binding():
    x = torch.zeros(16, device=DEV)
    y = torch.zeros(16, device=DEV, dtype=torch.bfloat16)
    with pytest.raises(smat.SmatError):
        smat.smat_simulate(x, y, y.clone(), dict(s=1.0, keep=2.0, sigma=0.0), 0, 0)
    with pytest.raises(smat.SmatError):
        smat.smat_simulate(x, y, x, dict(s=1.0, keep=1.0, sigma=0.0), 0, 0)   # out over theta
    with pytest.raises(smat.SmatError):
        smat.smat_backward_accum(x, x, dict(s=1.0, keep=1.0, sigma=0.0), 1.0, 0, 0)


def test_laplace_noise_parity():
    n = 1 << 20
    g = torch.Generator(DEV).manual_seed(12)
    theta = torch.randn(n, device=DEV, generator=g) * 0.02
    # keep = 0, sigma = 1 and theta0 = 0: the output is the unit Laplace draw itself
    zero = torch.zeros(n, device=DEV)
    out = torch.empty(n, device=DEV, dtype=torch.float32)
    p = dict(s=0.5, keep=0.0, sigma=1.0, rescale=1, noise_kind=oracle.NOISE_LAPLACE)
    smat.smat_simulate(theta, zero, out, p, 21, 4, 9)
    torch.cuda.synchronize()
    want = oracle.laplace_unit(21, 4, 9, 0, n)
    err = np.abs(out.cpu().numpy().astype(np.float64) - want)
    print(f"max |z_gpu - z| over {n} Laplace draws: {err.max():.3e}")
    assert err.max() <= Z_TOL
    # the full transform with a mask, bf16 and f32 outputs
    theta0 = (theta + torch.randn(n, device=DEV, generator=g) * 1e-3).to(torch.bfloat16)
    p = dict(s=0.8, keep=0.4, sigma=2e-3, rescale=1, noise_kind=oracle.NOISE_LAPLACE)
    for dt in (torch.bfloat16, torch.float32):
        o = torch.empty(n, device=DEV, dtype=dt)
        dist = compare_simulate(theta, theta0, o, p, 21, 5, 9, 8)
        if dist is not None:
            assert dist.max(initial=0) <= 1


def test_tensor_beyond_2_32_elements():
    # one tensor of 2^32 + 1029 elements: 64-bit element indices in both entry points, the last
    # chunk's ragged tail, and element offsets whose Philox group index exceeds 32 bits
    n = (1 << 32) + 1029
    theta = torch.empty(n, device=DEV, dtype=torch.float32)
    theta0 = torch.empty(n, device=DEV, dtype=torch.bfloat16)
    out = torch.empty(n, device=DEV, dtype=torch.bfloat16)
    g = torch.Generator(DEV).manual_seed(13)
    step_ = 1 << 28
    for a in range(0, n, step_):   # fill in slices to bound the temporaries
        b = min(n, a + step_)
        theta[a:b].normal_(0.0, 0.02, generator=g)
        theta0[a:b] = (theta[a:b] + torch.randn(b - a, device=DEV, generator=g) * 1e-3).to(torch.bfloat16)
    p = dict(s=0.6, keep=0.3, sigma=1e-3, rescale=1, noise_kind=0)
    seed, step, tid = 0x5EED1234, 9, 77
    smat.smat_simulate(theta, theta0, out, p, seed, step, tid)
    torch.cuda.synchronize()
    windows = [(0, 4096), ((1 << 31) - 17, (1 << 31) + 4099), ((1 << 32) - 2048, n)]
    for a, b in windows:
        th = theta[a:b].cpu().numpy()
        t0 = theta0[a:b].cpu().view(torch.int16).numpy().view(np.uint16)
        got = out[a:b].cpu().view(torch.int16).numpy().view(np.uint16)
        y, kept, eps = oracle.simulate_f64(th, t0, "bf16", p, seed, step, tid, a)
        coef = np.where(kept, oracle.coefficient(0.6, 0.3, 1), 0.0)
        ok, _ = check_theta_tilde(got, "bf16", y, th, oracle.as_f64(t0, "bf16"), coef, eps, 1e-3)
        assert ok.all(), f"window [{a},{b})"
    # the list entry point over the same tensor produces the same bytes
    out2 = torch.empty_like(out)
    with smat.Plan([theta], [out2], [theta0], tensor_ids=[tid]) as plan:
        plan.set_params([p])
        plan.simulate(seed, step)
        torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), out2.view(torch.int16))
    del theta, theta0, out, out2
    torch.cuda.empty_cache()
