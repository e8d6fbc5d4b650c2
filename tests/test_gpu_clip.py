"""GPU parity of the gradient-norm pass (smat_grad_norm_multi) and of norm clipping fed to the fused
optimizer step (grad_scale_dev of smat_adamw_fused / smat_adamw_fused_multi) against the oracle,
through the C ABI: ragged lists, misaligned tensors and offsets, accumulation, dropped tensors,
an empty list, determinism and argument errors."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_33437_amd as smat
import workloads
from helpers import host
from tolerances import SQNORM_ULPS, U, check_adam, check_sqnorm

pytestmark = pytest.mark.gpu
DEV = "cuda"
HP = dict(lr=2e-5, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-3, grad_scale=1.0, step=1)


def oracle_norm(gsn, gs_dt, params, lam, seed, step, ids, offs, accs=None):
    """(sumsq, sum of m^2) with m = |lambda t g~| + |acc| per element, in fp64."""
    sq, m2 = 0.0, 0.0
    for i in range(len(gsn)):
        acc = None if accs is None else accs[i]
        sq += oracle.grad_sqnorm(gsn[i], gs_dt, params[i], lam, seed, step, ids[i], offs[i], acc)
        m = np.abs(oracle.simulated_gradient(gsn[i], gs_dt, params[i], lam, seed, step, ids[i], offs[i]))
        if acc is not None:
            m = m + np.abs(np.asarray(acc, dtype=np.float64))
        m2 += float(np.dot(m, m))
    return sq, m2


def mini_plan():
    cfg = workloads.config("mini")
    inp = workloads.make_inputs(cfg, device="cpu")
    th = [t.to(DEV).view(-1) for t in inp.theta]
    t0 = [t.to(DEV) for t in inp.theta0]
    gs = [t.to(DEV) for t in inp.grad_sim]
    gt = [t.to(DEV) for t in inp.grad_theta]
    out = [torch.empty(t.numel(), dtype=torch.bfloat16, device=DEV) for t in th]
    return cfg, inp, (th, out, t0, gs, gt)


@pytest.mark.parametrize("accumulate", [False, True])
def test_list_norm_and_clip_factor(accumulate):
    cfg, inp, tensors = mini_plan()
    step = 7
    params = workloads.step_params(cfg, inp.settings, step)
    sumsq = torch.zeros(1, dtype=torch.float64, device=DEV)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    gsn = [host(g)[0] for g in inp.grad_sim]
    accs = [host(g)[0] for g in inp.grad_theta] if accumulate else None
    want, m2 = oracle_norm(gsn, "bf16", params, cfg.lam, cfg.smat_seed, step, list(range(cfg.count)),
                           [0] * cfg.count, accs)
    max_norm = 0.5 * math.sqrt(want)                       # clipping active
    with smat.Plan(*tensors) as plan:
        plan.set_params(params)
        plan.grad_norm(cfg.smat_seed, step, cfg.lam, accumulate, max_norm, sumsq, coef)
        torch.cuda.synchronize()
        got, got_coef = float(sumsq.item()), float(coef.item())
        assert check_sqnorm(got, want, m2), (got, want)
        want_coef = oracle.clip_coefficient(math.sqrt(want), max_norm)
        # coef = fl32(max_norm / (sqrt(sumsq) + 1e-6)): half the relative error of sumsq, plus roundings
        rel = 0.5 * SQNORM_ULPS * U * m2 / want + 2 * U
        assert abs(got_coef - want_coef) <= rel * want_coef
        # the same result on every call, and from the sumsq-only and factor-only forms
        again = torch.zeros_like(sumsq)
        plan.grad_norm(cfg.smat_seed, step, cfg.lam, accumulate, sumsq=again)
        c2 = torch.zeros_like(coef)
        plan.grad_norm(cfg.smat_seed, step, cfg.lam, accumulate, max_norm=max_norm, clip_coef=c2)
        plan.grad_norm(cfg.smat_seed, step, cfg.lam, accumulate, max_norm=1e30, clip_coef=coef)
        torch.cuda.synchronize()
        assert again.item() == got and c2.item() == got_coef
        assert coef.item() == 1.0                          # norm below max_norm: no clipping
    # the gradient tensors are read, never written
    for a, b in zip(tensors[3], inp.grad_sim):
        assert torch.equal(a.cpu().view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("g_dtype", [torch.bfloat16, torch.float32])
def test_misaligned_ragged_and_dropped_tensors(g_dtype):
    # sizes across several chunks with tails; tensors at odd element offsets within their buffers
    # (pointers off the quad alignment) and odd global offsets take the per-element path
    g = torch.Generator(DEV).manual_seed(3)
    sizes = [1, 3, 4, 5, 16384, 16385, 40000 + 3, 70001, 9001]
    shifts = [0, 1, 0, 3, 0, 0, 1, 0, 0]
    offs = [0, 0, 6, 0, 0, 2 ** 33 + 1, 4, 2 ** 34 + 8, 2 ** 34 - 4096]  # the last crosses 2^34 mid-tile
    keeps = [0.5, 0.0, 1.0, 0.3, 0.25, 0.5, 0.0, 0.7, 0.4]
    bufs = [torch.randn(n + 8, device=DEV, generator=g) for n in sizes]
    gs = [(b * 1e-2).to(g_dtype)[s:s + n] for b, s, n in zip(bufs, shifts, sizes)]
    gt = [(torch.randn(n + 8, device=DEV, generator=g) * 1e-3)[s:s + n] for s, n in zip(shifts, sizes)]
    th = [torch.zeros(n, device=DEV) for n in sizes]
    out = [torch.zeros(n, device=DEV, dtype=torch.bfloat16) for n in sizes]
    t0 = [torch.zeros(n, device=DEV, dtype=torch.bfloat16) for n in sizes]
    ids = [10 + i for i in range(len(sizes))]
    params = [dict(s=0.6, keep=k, sigma=0.0, rescale=1) for k in keeps]
    gsn = [host(x)[0] for x in gs]
    gs_dt = "bf16" if g_dtype == torch.bfloat16 else "f32"
    for accumulate in (False, True):
        accs = [host(x)[0] for x in gt] if accumulate else None
        want, m2 = oracle_norm(gsn, gs_dt, params, 0.5, 21, 9, ids, offs, accs)
        sumsq = torch.zeros(1, dtype=torch.float64, device=DEV)
        with smat.Plan(th, out, t0, gs, gt, tensor_ids=ids, elem_offsets=offs) as plan:
            plan.set_params(params)
            plan.grad_norm(21, 9, 0.5, accumulate, sumsq=sumsq)
            torch.cuda.synchronize()
        assert check_sqnorm(sumsq.item(), want, m2), (accumulate, sumsq.item(), want)


def test_empty_list_and_errors():
    sumsq = torch.full((1,), 7.0, dtype=torch.float64, device=DEV)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    with smat.Plan([], [], [], [], []) as plan:
        plan.set_params([])
        plan.grad_norm(1, 1, 1.0, False, 1.0, sumsq, coef)
        torch.cuda.synchronize()
        assert sumsq.item() == 0.0 and coef.item() == 1.0
    cfg, inp, tensors = mini_plan()
    with smat.Plan(*tensors) as plan:
        with pytest.raises(smat.SmatError):
            plan.grad_norm(1, 1, 1.0, sumsq=sumsq)                       # params never set
        plan.set_params(workloads.step_params(cfg, inp.settings, 3))
        with pytest.raises(smat.SmatError):
            plan.grad_norm(1, 1, 1.0)                                    # no output
        with pytest.raises(smat.SmatError):
            plan.grad_norm(1, 1, 1.0, max_norm=0.0, clip_coef=coef)      # bad max_norm
        with pytest.raises(smat.SmatError):
            plan.grad_norm(1, 1, float("nan"), sumsq=sumsq)
        with pytest.raises(smat.SmatError):
            plan.grad_norm(1, 1, 1.0, sumsq=coef)                        # wrong dtype for sumsq


@pytest.mark.parametrize("accumulate", [False, True])
def test_clipped_fused_adamw_list(accumulate):
    cfg, inp, tensors = mini_plan()
    th, out, t0, gs, gt = tensors
    gen = torch.Generator(DEV).manual_seed(8)
    m1 = [torch.randn(t.numel(), device=DEV, generator=gen) * 1e-3 for t in th]
    m2 = [torch.rand(t.numel(), device=DEV, generator=gen) * 1e-6 for t in th]
    old = [(host(a)[0], host(b)[0], host(c)[0]) for a, b, c in zip(th, m1, m2)]
    step = 11
    params = workloads.step_params(cfg, inp.settings, step)
    hp = dict(HP, step=4, grad_scale=0.5)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    with smat.Plan(*tensors) as plan:
        plan.set_params(params)
        plan.bind_adam_state(m1, m2)
        plan.grad_norm(cfg.smat_seed, step, cfg.lam, accumulate, max_norm=1e-3, clip_coef=coef)
        plan.adamw_fused(cfg.smat_seed, step, cfg.lam, hp, accumulate=accumulate, grad_scale_dev=coef)
        torch.cuda.synchronize()
    c = float(coef.item())
    assert 0.0 < c < 1.0
    hp_o = dict(hp, grad_scale=float(np.float32(hp["grad_scale"])) * c)   # the kernel's fl(grad_scale * c)
    for i in range(cfg.count):
        acc = host(inp.grad_theta[i])[0] if accumulate else None
        gsn = host(inp.grad_sim[i])[0]
        _, f64 = oracle.adamw_fused(gsn, "bf16", *old[i], params[i], cfg.lam, hp_o, cfg.smat_seed, step, i,
                                    grad_acc=acc)
        gmag = np.abs(oracle.simulated_gradient(gsn, "bf16", params[i], cfg.lam, cfg.smat_seed, step, i))
        if acc is not None:
            gmag = gmag + np.abs(acc.astype(np.float64))
        gmag = gmag * abs(hp_o["grad_scale"])
        got = (host(th[i])[0], host(m1[i])[0], host(m2[i])[0])
        for name, ok in zip(("theta", "exp_avg", "exp_avg_sq"), check_adam(got, old[i], f64, hp_o, gmag)):
            assert ok.all(), f"tensor {i} {name}: {np.count_nonzero(~ok)} mismatches"


def test_single_tensor_device_scale():
    n = 100003
    g = torch.Generator(DEV).manual_seed(12)
    th = torch.randn(n, device=DEV, generator=g) * 0.02
    m1, m2 = torch.zeros(n, device=DEV), torch.zeros(n, device=DEV)
    gs = (torch.randn(n, device=DEV, generator=g) * 1e-2).to(torch.bfloat16)
    p = dict(s=0.6, keep=0.3, sigma=0.0, rescale=1)
    scale = torch.tensor([0.37], dtype=torch.float32, device=DEV)
    hp = dict(HP, step=2, grad_scale=2.0)
    old = (host(th)[0], host(m1)[0], host(m2)[0])
    smat.smat_adamw_fused(gs, th, m1, m2, p, 0.5, hp, 5, 3, 1, grad_scale_dev=scale)
    torch.cuda.synchronize()
    hp_o = dict(hp, grad_scale=2.0 * float(np.float32(0.37)))
    gsn = host(gs)[0]
    _, f64 = oracle.adamw_fused(gsn, "bf16", *old, p, 0.5, hp_o, 5, 3, 1)
    got = (host(th)[0], host(m1)[0], host(m2)[0])
    assert all(ok.all() for ok in check_adam(got, old, f64, hp_o))
    with pytest.raises(smat.SmatError):
        smat.smat_adamw_fused(gs, th, m1, m2, p, 0.5, hp, 5, 3, 1, grad_scale_dev=scale.double())
