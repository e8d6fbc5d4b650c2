"""GPU parity of the fused optimizer step (smat_adamw_fused, smat_adamw_fused_multi) against the
oracle's AdamW fed by the simulated-loss gradient, through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_33437_amd as smat
import workloads
from helpers import host
from tolerances import check_adam

pytestmark = pytest.mark.gpu
DEV = "cuda"
HP = dict(lr=2e-5, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-3, grad_scale=1.0, step=1)


def _state(n, g, shift=0):
    th = (torch.randn(n + 8, device=DEV, generator=g) * 0.02)[shift:shift + n]
    m1 = (torch.randn(n + 8, device=DEV, generator=g) * 1e-3)[shift:shift + n]
    m2 = (torch.rand(n + 8, device=DEV, generator=g) * 1e-6)[shift:shift + n]
    return th, m1, m2


def _check(th, m1, m2, old, gsn, gs_dt, p, lam, hp, seed, step, tid, off, acc=None):
    (_, _, _), f64 = oracle.adamw_fused(gsn, gs_dt, old[0], old[1], old[2], p, lam, hp, seed, step, tid, off,
                                         grad_acc=acc)
    gmag = np.abs(oracle.simulated_gradient(gsn, gs_dt, p, lam, seed, step, tid, off, None, hp["grad_scale"]))
    if acc is not None:
        gmag = gmag + abs(float(np.float32(hp["grad_scale"]))) * np.abs(np.asarray(acc, dtype=np.float64))
    ok = check_adam((host(th)[0], host(m1)[0], host(m2)[0]), old, f64, hp, gmag)
    for name, o in zip(("theta", "exp_avg", "exp_avg_sq"), ok):
        bad = np.flatnonzero(~o)
        assert bad.size == 0, f"{name}: {bad.size} mismatches, first {bad[:5]}"


@pytest.mark.parametrize("n,shift,off", [(1, 0, 0), (5, 0, 0), (4096, 0, 0), (100003, 0, 0), (50001, 1, 3),
                                          (70000, 0, 2 ** 34 + 8), (5000, 0, 2 ** 34 - 1000)])
@pytest.mark.parametrize("g_dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("accumulate", [False, True])
def test_single_tensor(n, shift, off, g_dtype, accumulate):
    g = torch.Generator(DEV).manual_seed(n + shift)
    th, m1, m2 = _state(n, g, shift)
    gs = (torch.randn(n + 8, device=DEV, generator=g) * 1e-2).to(g_dtype)[shift:shift + n]
    acc = (torch.randn(n + 8, device=DEV, generator=g) * 1e-3)[shift:shift + n] if accumulate else None
    p = dict(s=0.6, keep=0.3, sigma=1e-3, rescale=1, noise_kind=0)
    hp = dict(HP, step=3, grad_scale=0.75)
    old = (host(th)[0], host(m1)[0], host(m2)[0])
    gsn, gs_dt = host(gs)
    accn = host(acc)[0] if accumulate else None
    smat.smat_adamw_fused(gs, th, m1, m2, p, 0.5, hp, 99, 7, 5, off, grad_acc=acc)
    torch.cuda.synchronize()
    _check(th, m1, m2, old, gsn, gs_dt, p, 0.5, hp, 99, 7, 5, off, accn)
    if accumulate:   # the accumulator is read, never written
        assert torch.equal(acc.cpu(), torch.from_numpy(accn))


def test_several_steps_and_degenerate_masks():
    n = 65536 + 3
    g = torch.Generator(DEV).manual_seed(4)
    th, m1, m2 = (torch.randn(n, device=DEV, generator=g) * 0.02, torch.zeros(n, device=DEV),
                  torch.zeros(n, device=DEV))
    for k, keep in zip((1, 2, 3, 4), (0.5, 1.0, 0.0, 0.2)):
        gs = (torch.randn(n, device=DEV, generator=g) * 1e-2).to(torch.bfloat16)
        p = dict(s=0.8, keep=keep, sigma=0.0, rescale=1, noise_kind=0)
        hp = dict(HP, step=k, weight_decay=0.1)
        old = (host(th)[0], host(m1)[0], host(m2)[0])
        smat.smat_adamw_fused(gs, th, m1, m2, p, 1.0, hp, 3, 100 + k, 1)
        torch.cuda.synchronize()
        _check(th, m1, m2, old, host(gs)[0], "bf16", p, 1.0, hp, 3, 100 + k, 1, 0)


def test_matches_backward_then_torch_adamw():
    # fused == smat_backward_accum into a zero gradient followed by torch's AdamW (fp32 on the GPU)
    n = 1 << 18
    g = torch.Generator(DEV).manual_seed(6)
    th = torch.randn(n, device=DEV, generator=g) * 0.02
    gs = (torch.randn(n, device=DEV, generator=g) * 1e-2).to(torch.bfloat16)
    p = dict(s=0.7, keep=0.25, sigma=1e-3)
    hp = dict(HP, lr=1e-3)
    param = torch.nn.Parameter(th.clone())
    grad = torch.zeros(n, device=DEV)
    smat.smat_backward_accum(gs, grad, p, 0.5, 11, 3, 2)
    param.grad = grad
    f32 = lambda x: float(np.float32(x))   # the ABI carries the hyperparameters as fp32
    opt = torch.optim.AdamW([param], lr=f32(hp["lr"]), betas=(f32(0.9), f32(0.999)), eps=f32(1e-8),
                            weight_decay=f32(1e-3), foreach=False)
    opt.step()
    m1, m2 = torch.zeros(n, device=DEV), torch.zeros(n, device=DEV)
    smat.smat_adamw_fused(gs, th, m1, m2, p, 0.5, hp, 11, 3, 2)
    torch.cuda.synchronize()
    st = opt.state[param]
    torch.testing.assert_close(th, param.detach(), rtol=1e-5, atol=1e-9)
    torch.testing.assert_close(m1, st["exp_avg"], rtol=1e-5, atol=1e-12)
    torch.testing.assert_close(m2, st["exp_avg_sq"], rtol=1e-5, atol=1e-16)


@pytest.mark.parametrize("accumulate", [False, True])
def test_plan_matches_oracle_and_needs_expert_storage(accumulate):
    cfg = workloads.config("mini")
    inp = workloads.make_inputs(cfg, device="cpu")
    th = [t.to(DEV).view(-1) for t in inp.theta]
    t0 = [t.to(DEV) for t in inp.theta0]
    gs = [t.to(DEV) for t in inp.grad_sim]
    gt = [t.to(DEV) for t in inp.grad_theta]
    out = [torch.empty(t.numel(), dtype=torch.bfloat16, device=DEV) for t in th]
    gen = torch.Generator(DEV).manual_seed(8)
    m1 = [torch.randn(t.numel(), device=DEV, generator=gen) * 1e-3 for t in th]
    m2 = [torch.rand(t.numel(), device=DEV, generator=gen) * 1e-6 for t in th]
    old = [(host(a)[0], host(b)[0], host(c)[0]) for a, b, c in zip(th, m1, m2)]
    step = 3
    params = workloads.step_params(cfg, inp.settings, step)
    hp = dict(HP, step=5)
    with smat.Plan(th, out, t0, gs, gt) as plan:
        plan.set_params(params)
        with pytest.raises(smat.SmatError):
            plan.adamw_fused(cfg.smat_seed, step, cfg.lam, hp)          # no optimizer state yet
        plan.bind_adam_state(m1, m2)
        plan.simulate(cfg.smat_seed, step)
        plan.switch_storage(smat.SMAT_SIMULATED)
        with pytest.raises(smat.SmatError):
            plan.adamw_fused(cfg.smat_seed, step, cfg.lam, hp)          # simulated storage active
        plan.switch_storage(smat.SMAT_EXPERT)
        plan.adamw_fused(cfg.smat_seed, step, cfg.lam, hp, accumulate=accumulate)
        torch.cuda.synchronize()
    for i in range(cfg.count):
        acc = host(inp.grad_theta[i])[0].ravel() if accumulate else None
        _check(th[i], m1[i], m2[i], old[i], host(inp.grad_sim[i])[0].ravel(), "bf16", params[i], cfg.lam, hp,
               cfg.smat_seed, step, i, 0, acc)


@pytest.mark.parametrize("accumulate", [False, True])
def test_plan_tiles_across_a_high_counter_word_boundary(accumulate):
    # global offsets just below multiples of 2^34 elements: one tile of each tensor crosses the
    # change of the group index's high word
    g = torch.Generator(DEV).manual_seed(35)
    sizes, offs, ids = [5000, 20001], [2 ** 34 - 1000, 2 ** 35 - 8192], [6, 7]
    states = [_state(n, g) for n in sizes]
    th = [s[0] for s in states]
    gs = [(torch.randn(n, device=DEV, generator=g) * 1e-2).to(torch.bfloat16) for n in sizes]
    acc = [torch.randn(n, device=DEV, generator=g) * 1e-3 for n in sizes]
    out = [torch.empty(n, dtype=torch.bfloat16, device=DEV) for n in sizes]
    old = [tuple(host(x)[0] for x in s) for s in states]
    params = [dict(s=0.6, keep=0.3, sigma=0.0, rescale=1), dict(s=0.8, keep=0.5, sigma=0.0, rescale=1)]
    hp = dict(HP, step=4, grad_scale=0.5)
    t0 = [x.to(torch.bfloat16) for x in th]
    with smat.Plan(th, out, t0, gs, acc, tensor_ids=ids, elem_offsets=offs) as plan:
        plan.set_params(params)
        plan.bind_adam_state([s[1] for s in states], [s[2] for s in states])
        plan.adamw_fused(21, 6, 0.5, hp, accumulate=accumulate)
        torch.cuda.synchronize()
    for i in range(len(sizes)):
        _check(*states[i], old[i], host(gs[i])[0], "bf16", params[i], 0.5, hp, 21, 6, ids[i], offs[i],
               host(acc[i])[0] if accumulate else None)


def test_bind_adam_state_rejects_moments_over_theta0_or_buffer():
    # the optimizer step writes the moments: they must not alias theta0 (resident mode) or the buffer
    n = 4096
    th = torch.zeros(n, device=DEV)
    t0_store = torch.zeros(2 * n, dtype=torch.bfloat16, device=DEV)    # theta0 = its first n entries
    out_store = torch.zeros(2 * n, dtype=torch.bfloat16, device=DEV)   # buffer = its first n entries
    gs = torch.zeros(n, dtype=torch.bfloat16, device=DEV)
    m2 = torch.zeros(n, device=DEV)
    with smat.Plan([th], [out_store[:n]], [t0_store[:n]], [gs], None) as plan:
        for bad in (t0_store.view(torch.float32), out_store.view(torch.float32)):   # n floats each
            with pytest.raises(smat.SmatError, match="INVALID"):
                plan.bind_adam_state([bad], [m2])
            with pytest.raises(smat.SmatError, match="INVALID"):
                plan.bind_adam_state([m2.clone()], [bad])
        plan.bind_adam_state([torch.zeros(n, device=DEV)], [m2])      # disjoint arrays are accepted
