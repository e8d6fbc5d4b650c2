"""GPU tests of the device-driven list calls (smat_simulate_multi_dev, smat_backward_multi_dev,
smat_grad_norm_multi_dev, smat_adamw_fused_multi_dev), through the C ABI: they give the bits of the
host-driven calls for s' = fl32(scale * s) (and the same learning rate and optimizer step), agree
with the oracle, and serve every step from one HIP graph (torch.cuda.CUDAGraph stream capture)
whether the step state is rewritten from the host between replays or advanced by torch ops captured
in the same graph; every replay is checked against the eager host-driven result of its step."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_33437_amd as smat
import workloads
from helpers import host
from tolerances import check_adam, check_grad, check_theta_tilde

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def mini():
    cfg = workloads.config("mini")
    inp = workloads.make_inputs(cfg, device="cpu")
    return cfg, inp


def base_params(cfg, inp, step):
    """The mini list's per-tensor settings, with rescale off on one masked tensor, a tensor that keeps
    nothing (and has no noise) and Laplace noise on another: every form of the coefficient."""
    p = workloads.step_params(cfg, inp.settings, step)
    p[2] = dict(p[2], rescale=0)
    p[5] = dict(p[5], keep=0.0, sigma=0.0)
    p[7] = dict(p[7], noise_kind=smat.SMAT_NOISE_LAPLACE, sigma=1e-4)
    return p


def scaled(params, scale):
    """The host-driven parameters of a device step: s' = fl32(scale * s) per tensor."""
    return [dict(p, s=float(np.float32(scale) * np.float32(p["s"]))) for p in params]


def list_tensors(inp):
    th = [t.to(DEV).view(-1) for t in inp.theta]
    t0 = [t.to(DEV).view(-1) for t in inp.theta0]
    gs = [t.to(DEV).view(-1) for t in inp.grad_sim]
    return th, t0, gs


def fresh(inp):
    out = [torch.full((t.numel(),), float("nan"), dtype=torch.bfloat16, device=DEV) for t in inp.theta]
    gt = [t.to(DEV).view(-1).clone() for t in inp.grad_theta]
    return out, gt


def same_bits(a, b):
    return all(torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x.view(torch.int32),
                           y.view(torch.int16) if y.dtype == torch.bfloat16 else y.view(torch.int32))
               for x, y in zip(a, b))


@pytest.mark.parametrize("accumulate", [True, False])
def test_device_step_is_host_step_with_scaled_s(mini, accumulate):
    cfg, inp = mini
    th, t0, gs = list_tensors(inp)
    out_d, gt_d = fresh(inp)
    out_h, gt_h = fresh(inp)
    step, scale = 5, 0.8125
    base = base_params(cfg, inp, step)
    state = smat.StepState(cfg.smat_seed, step, scale)
    with smat.Plan(th, out_d, t0, gs, gt_d) as pd, smat.Plan(th, out_h, t0, gs, gt_h) as ph:
        pd.set_params(base)
        pd.simulate_dev(state)
        pd.backward_dev(state, cfg.lam, accumulate)
        ph.set_params(scaled(base, scale))
        ph.simulate(cfg.smat_seed, step)
        ph.backward(cfg.smat_seed, step, cfg.lam, accumulate)
        torch.cuda.synchronize()
    assert same_bits(out_d, out_h)
    assert same_bits(gt_d, gt_h)


def test_device_step_oracle_parity(mini):
    cfg, inp = mini
    th, t0, gs = list_tensors(inp)
    out, gt = fresh(inp)
    step, scale = 9, 0.4375
    base = base_params(cfg, inp, step)
    params = scaled(base, scale)
    state = smat.StepState(cfg.smat_seed, step, scale)
    with smat.Plan(th, out, t0, gs, gt) as plan:
        plan.set_params(base)
        plan.simulate_dev(state)
        plan.backward_dev(state, cfg.lam, True)
        torch.cuda.synchronize()
    for i in range(cfg.count):
        p = params[i]
        thn, _ = host(inp.theta[i])
        t0n, t0_dt = host(inp.theta0[i])
        y, kept, eps = oracle.simulate_f64(thn.ravel(), t0n.ravel(), t0_dt, p, cfg.smat_seed, step, i)
        coef = np.where(kept, oracle.coefficient(p["s"], p["keep"], p["rescale"]), 0.0)
        got, out_dt = host(out[i])
        ok, _ = check_theta_tilde(got, out_dt, y, thn.ravel(), oracle.as_f64(t0n.ravel(), t0_dt), coef, eps,
                                  p["sigma"])
        assert ok.all(), f"tensor {i}: {np.count_nonzero(~ok)} theta~ mismatches"
        gsn, gs_dt = host(inp.grad_sim[i])
        g_old, _ = host(inp.grad_theta[i])
        want = oracle.backward_accum(gsn.ravel(), gs_dt, g_old.ravel(), p, cfg.lam, cfg.smat_seed, step, i)
        gotg, _ = host(gt[i])
        incr = np.abs(cfg.lam * coef * oracle.as_f64(gsn.ravel(), gs_dt))
        assert check_grad(gotg.ravel(), want, g_old.ravel(), incr).all(), f"tensor {i}"
    assert (host(out[5])[0] == host(inp.theta0[5])[0].ravel()).all()    # keep = 0, no noise: theta0


@pytest.mark.parametrize("g_dtype", [torch.bfloat16, torch.float32])
def test_device_step_ragged_misaligned(g_dtype):
    # per-element paths: pointers off the quad alignment, odd offsets, a tile that crosses 2^34
    g = torch.Generator(DEV).manual_seed(4)
    sizes = [1, 5, 16385, 70001, 9001, 40003]
    shifts = [0, 3, 0, 1, 0, 2]
    offs = [0, 0, 2 ** 33 + 1, 4, 2 ** 34 - 4096, 2 ** 34 + 8]
    keeps = [0.5, 1.0, 0.25, 0.0, 0.4, 0.7]
    th = [(torch.randn(n + 8, device=DEV, generator=g) * 0.02)[s:s + n] for n, s in zip(sizes, shifts)]
    t0 = [(torch.randn(n + 8, device=DEV, generator=g) * 0.02)[s:s + n] for n, s in zip(sizes, shifts)]
    gs = [(torch.randn(n + 8, device=DEV, generator=g) * 1e-2).to(g_dtype)[s:s + n] for n, s in zip(sizes, shifts)]
    gt0 = [(torch.randn(n + 8, device=DEV, generator=g) * 1e-3)[s:s + n] for n, s in zip(sizes, shifts)]
    ids = [20 + i for i in range(len(sizes))]
    base = [dict(s=0.25 + 0.125 * i, keep=k, sigma=1e-3 * (i % 2), rescale=1, noise_kind=i % 3)
            for i, k in enumerate(keeps)]
    step, scale = 1 << 29, 0.6
    res = {}
    for mode in ("dev", "host"):
        out = [torch.full((n,), float("nan"), device=DEV) for n in sizes]
        gt = [x.clone() for x in gt0]
        with smat.Plan(th, out, t0, gs, gt, tensor_ids=ids, elem_offsets=offs,
                       dtypes=(smat.SMAT_F32, smat.SMAT_F32, smat.SMAT_BF16 if g_dtype == torch.bfloat16
                               else smat.SMAT_F32)) as plan:
            if mode == "dev":
                state = smat.StepState(77, step, scale)
                plan.set_params(base)
                plan.simulate_dev(state)
                plan.backward_dev(state, 0.5, True)
            else:
                plan.set_params(scaled(base, scale))
                plan.simulate(77, step)
                plan.backward(77, step, 0.5, True)
            torch.cuda.synchronize()
        res[mode] = (out, gt)
    assert same_bits(res["dev"][0], res["host"][0])
    assert same_bits(res["dev"][1], res["host"][1])


def test_step_state_views():
    st = smat.StepState((1 << 40) + 5, 123, 0.25)
    assert st.seed_view.item() == (1 << 40) + 5
    assert st.step_view.item() == 123
    assert st.scale_view.item() == 0.25
    st.step_view.add_(2)
    st.scale_view.mul_(3.0)
    assert st.step_view.item() == 125 and st.scale_view.item() == 0.75


@pytest.mark.parametrize("accumulate", [False, True])
def test_graph_replays_with_host_written_state(mini, accumulate):
    cfg, inp = mini
    th, t0, gs = list_tensors(inp)
    out_d, gt_d = fresh(inp)
    out_h, gt_h = fresh(inp)
    base = base_params(cfg, inp, 0)
    state = smat.StepState(cfg.smat_seed, 0, 1.0)
    steps = [(cfg.smat_seed, 3, 0.5), (cfg.smat_seed + 1, 4, 0.9), (cfg.smat_seed, 1 << 20, 0.3125)]
    gen = torch.Generator(DEV).manual_seed(6)
    with smat.Plan(th, out_d, t0, gs, gt_d) as pd, smat.Plan(th, out_h, t0, gs, gt_h) as ph:
        pd.set_params(base)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):                     # one eager call before capture
            pd.simulate_dev(state)
            pd.backward_dev(state, cfg.lam, accumulate)
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            pd.simulate_dev(state)
            pd.backward_dev(state, cfg.lam, accumulate)
        for seed, step, scale in steps:
            # eager work between replays: fresh gradients in both lists, poisoned outputs
            for a, b in zip(gt_d, gt_h):
                a.copy_(torch.randn(a.numel(), device=DEV, generator=gen) * 1e-3)
                b.copy_(a)
            for o in out_d:
                o.fill_(float("nan"))
            state.set(seed, step, scale)
            graph.replay()
            ph.set_params(scaled(base, scale))
            ph.simulate(seed, step)
            ph.backward(seed, step, cfg.lam, accumulate)
            torch.cuda.synchronize()
            assert same_bits(out_d, out_h), (seed, step, scale)
            assert same_bits(gt_d, gt_h), (seed, step, scale)
        del graph


def test_graph_advances_its_own_state(mini):
    cfg, inp = mini
    th, t0, gs = list_tensors(inp)
    out_d, gt_d = fresh(inp)
    out_h, gt_h = fresh(inp)
    base = base_params(cfg, inp, 0)
    step0, scale0 = 40, 0.75
    state = smat.StepState(cfg.smat_seed, step0, scale0)
    with smat.Plan(th, out_d, t0, gs, gt_d) as pd, smat.Plan(th, out_h, t0, gs, gt_h) as ph:
        pd.set_params(base)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):                     # warm the torch ops and the plan once
            state.step_view.add_(1)
            state.scale_view.mul_(0.5)
            pd.simulate_dev(state)
            pd.backward_dev(state, cfg.lam, False)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        state.set(cfg.smat_seed, step0, scale0)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            state.step_view.add_(1)
            state.scale_view.mul_(0.5)
            pd.simulate_dev(state)
            pd.backward_dev(state, cfg.lam, False)
        for k in range(1, 4):
            for o in out_d:
                o.fill_(float("nan"))
            graph.replay()
            step, scale = step0 + k, scale0 * 0.5 ** k
            ph.set_params(scaled(base, scale))
            ph.simulate(cfg.smat_seed, step)
            ph.backward(cfg.smat_seed, step, cfg.lam, False)
            torch.cuda.synchronize()
            assert state.step_view.item() == step and state.scale_view.item() == scale
            assert same_bits(out_d, out_h), k
            assert same_bits(gt_d, gt_h), k
        del graph


def test_device_calls_errors(mini):
    cfg, inp = mini
    th, t0, gs = list_tensors(inp)
    out, gt = fresh(inp)
    state = smat.StepState(1, 2, 0.5)
    with smat.Plan(th, out, t0, gs, gt) as plan:
        with pytest.raises(smat.SmatError):
            plan.simulate_dev(state)                                   # parameters never set
        plan.set_params(base_params(cfg, inp, 2))
        with pytest.raises(smat.SmatError):
            plan.simulate_dev(torch.zeros(3, dtype=torch.int32, device=DEV))   # 12 bytes
        with pytest.raises(smat.SmatError):
            plan.simulate_dev(torch.zeros(4, dtype=torch.int32))               # host tensor
        with pytest.raises(smat.SmatError):
            plan.simulate_dev(torch.zeros(8, dtype=torch.int32, device=DEV)[1:5])  # not 16-byte aligned
        with pytest.raises(smat.SmatError):
            plan.backward_dev(state, float("inf"))
        plan.simulate_dev(state.tensor)                                # a plain 16-byte tensor works too
        plan.switch_storage(smat.SMAT_SIMULATED)
        with pytest.raises(smat.SmatError):
            plan.simulate_dev(state)                                   # simulated storage active
        plan.backward_dev(state, cfg.lam)                              # the backward needs no switch
        plan.switch_storage(smat.SMAT_EXPERT)
        torch.cuda.synchronize()
    hosts = [t.contiguous().view(-1).pin_memory() for t in inp.theta0]
    bufs = [torch.zeros(t.numel(), dtype=torch.bfloat16, device=DEV) for t in th]
    with smat.Plan(th, bufs, None, offload=True, theta0_hosts=hosts,
                   dtypes=(smat.SMAT_BF16, smat.SMAT_BF16, smat.SMAT_BF16)) as off:
        off.set_params(base_params(cfg, inp, 2))
        with pytest.raises(smat.SmatError, match="offload"):
            off.simulate_dev(state)
        torch.cuda.synchronize()


# ---------------------------------------------------------------- optimizer step and gradient norm
HP = dict(beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-3, grad_scale=0.5)


def adam_twin(inp, seed):
    """theta and the two moments of every tensor, twice (one set per plan), equal bit for bit."""
    gen = torch.Generator(DEV).manual_seed(seed)
    th = [t.to(DEV).view(-1).clone() for t in inp.theta]
    m1 = [torch.randn(t.numel(), device=DEV, generator=gen) * 1e-3 for t in th]
    m2 = [torch.rand(t.numel(), device=DEV, generator=gen) * 1e-6 for t in th]
    return (th, m1, m2), tuple([x.clone() for x in xs] for xs in (th, m1, m2))


@pytest.mark.parametrize("accumulate", [False, True])
def test_device_norm_is_host_norm(mini, accumulate):
    cfg, inp = mini
    th, t0, gs = list_tensors(inp)
    out, gt = fresh(inp)
    step, scale = 6, 0.6875
    base = base_params(cfg, inp, step)
    state = smat.StepState(cfg.smat_seed, step, scale)
    sq_d, sq_h = (torch.zeros(1, dtype=torch.float64, device=DEV) for _ in range(2))
    c_d, c_h = (torch.zeros(1, dtype=torch.float32, device=DEV) for _ in range(2))
    with smat.Plan(th, out, t0, gs, gt) as plan:
        plan.set_params(base)
        plan.grad_norm_dev(state, cfg.lam, accumulate, 1e-3, sq_d, c_d)
        plan.set_params(scaled(base, scale))
        plan.grad_norm(cfg.smat_seed, step, cfg.lam, accumulate, 1e-3, sq_h, c_h)
        torch.cuda.synchronize()
    assert sq_d.item() > 0 and 0 < c_d.item() < 1
    assert torch.equal(sq_d.view(torch.int64), sq_h.view(torch.int64))
    assert torch.equal(c_d.view(torch.int32), c_h.view(torch.int32))


@pytest.mark.parametrize("accumulate,clip", [(False, False), (True, False), (False, True), (True, True)])
def test_device_adamw_is_host_adamw(mini, accumulate, clip):
    cfg, inp = mini
    _, t0, gs = list_tensors(inp)
    (th_d, m1_d, m2_d), (th_h, m1_h, m2_h) = adam_twin(inp, 8)
    out_d, gt = fresh(inp)
    out_h, _ = fresh(inp)
    step, scale, lr, k = 11, 0.8125, 2e-5, 7
    base = base_params(cfg, inp, step)
    state, adam = smat.StepState(cfg.smat_seed, step, scale), smat.AdamStepState(lr, k)
    coef = torch.tensor([0.37], dtype=torch.float32, device=DEV) if clip else None
    with smat.Plan(th_d, out_d, t0, gs, gt) as pd, smat.Plan(th_h, out_h, t0, gs, gt) as ph:
        pd.set_params(base)
        pd.bind_adam_state(m1_d, m2_d)
        pd.adamw_fused_dev(state, adam, cfg.lam, HP, accumulate, coef)
        ph.set_params(scaled(base, scale))
        ph.bind_adam_state(m1_h, m2_h)
        ph.adamw_fused(cfg.smat_seed, step, cfg.lam, dict(HP, lr=lr, step=k), accumulate, coef)
        torch.cuda.synchronize()
    for a, b in ((th_d, th_h), (m1_d, m1_h), (m2_d, m2_h)):
        assert same_bits(a, b)


def test_device_adamw_oracle_parity(mini):
    cfg, inp = mini
    _, t0, gs = list_tensors(inp)
    (th, m1, m2), _ = adam_twin(inp, 9)
    out, gt = fresh(inp)
    old = [(host(a)[0], host(b)[0], host(c)[0]) for a, b, c in zip(th, m1, m2)]
    step, scale, lr, k = 13, 0.5625, 3e-5, 4
    base = base_params(cfg, inp, step)
    params = scaled(base, scale)
    with smat.Plan(th, out, t0, gs, gt) as plan:
        plan.set_params(base)
        plan.bind_adam_state(m1, m2)
        plan.adamw_fused_dev(smat.StepState(cfg.smat_seed, step, scale), smat.AdamStepState(lr, k), cfg.lam, HP)
        torch.cuda.synchronize()
    hp = dict(HP, lr=lr, step=k)
    for i in range(cfg.count):
        gsn = host(inp.grad_sim[i])[0]
        _, f64 = oracle.adamw_fused(gsn, "bf16", *old[i], params[i], cfg.lam, hp, cfg.smat_seed, step, i)
        gmag = np.abs(oracle.simulated_gradient(gsn, "bf16", params[i], cfg.lam, cfg.smat_seed, step, i)) * hp["grad_scale"]
        got = (host(th[i])[0], host(m1[i])[0], host(m2[i])[0])
        for name, ok in zip(("theta", "exp_avg", "exp_avg_sq"), check_adam(got, old[i], f64, hp, gmag)):
            assert ok.all(), f"tensor {i} {name}: {np.count_nonzero(~ok)} mismatches"


@pytest.mark.parametrize("accumulate", [False, True])
def test_graph_of_a_clipped_fused_step(mini, accumulate):
    """simulate, gradient norm and clipped fused update captured once; each replay advances the SMAT
    step and the optimizer step on the device and matches the host-driven step on twin tensors."""
    cfg, inp = mini
    _, t0, gs = list_tensors(inp)
    (th_d, m1_d, m2_d), (th_h, m1_h, m2_h) = adam_twin(inp, 10)
    out_d, gt = fresh(inp)
    out_h, _ = fresh(inp)
    base = base_params(cfg, inp, 0)
    step0, scale, lr, k0, max_norm = 20, 0.75, 1e-4, 3, 2e-3
    state, adam = smat.StepState(cfg.smat_seed, step0, scale), smat.AdamStepState(lr, k0)
    c_d, c_h = (torch.zeros(1, dtype=torch.float32, device=DEV) for _ in range(2))
    with smat.Plan(th_d, out_d, t0, gs, gt) as pd, smat.Plan(th_h, out_h, t0, gs, gt) as ph:
        pd.set_params(base)
        pd.bind_adam_state(m1_d, m2_d)
        ph.bind_adam_state(m1_h, m2_h)

        def step_ops():
            state.step_view.add_(1)
            adam.step_view.add_(1)
            pd.simulate_dev(state)
            pd.grad_norm_dev(state, cfg.lam, accumulate, max_norm, clip_coef=c_d)
            pd.adamw_fused_dev(state, adam, cfg.lam, HP, accumulate, c_d)

        # warm the torch ops once on a side stream on scratch states, then capture
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            smat.StepState(0, 0, 1.0).step_view.add_(1)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step_ops()
        torch.cuda.synchronize()
        # capture ran nothing: the tensors and states are as they were
        assert state.step_view.item() == step0 and adam.step_view.item() == k0
        for r in range(1, 4):
            for o in out_d:
                o.fill_(float("nan"))
            graph.replay()
            step, k = step0 + r, k0 + r
            ph.set_params(scaled(base, scale))
            ph.simulate(cfg.smat_seed, step)
            ph.grad_norm(cfg.smat_seed, step, cfg.lam, accumulate, max_norm, clip_coef=c_h)
            ph.adamw_fused(cfg.smat_seed, step, cfg.lam, dict(HP, lr=lr, step=k), accumulate, c_h)
            torch.cuda.synchronize()
            assert 0 < c_d.item() < 1 and c_d.item() == c_h.item(), r
            assert same_bits(out_d, out_h), r
            for a, b in ((th_d, th_h), (m1_d, m1_h), (m2_d, m2_h)):
                assert same_bits(a, b), r
        del graph


def test_device_optimizer_errors(mini):
    cfg, inp = mini
    _, t0, gs = list_tensors(inp)
    (th, m1, m2), _ = adam_twin(inp, 11)
    out, gt = fresh(inp)
    state, adam = smat.StepState(1, 2, 0.5), smat.AdamStepState(1e-4, 1)
    sq = torch.zeros(1, dtype=torch.float64, device=DEV)
    with smat.Plan(th, out, t0, gs, gt) as plan:
        plan.set_params(base_params(cfg, inp, 2))
        with pytest.raises(smat.SmatError):
            plan.adamw_fused_dev(state, adam, cfg.lam, HP)                      # optimizer state never bound
        plan.bind_adam_state(m1, m2)
        with pytest.raises(smat.SmatError):
            plan.adamw_fused_dev(state, adam, cfg.lam, dict(HP, beta1=1.0))    # bad hyperparameter
        with pytest.raises(smat.SmatError):
            plan.adamw_fused_dev(state, torch.zeros(4, dtype=torch.int32, device=DEV), cfg.lam, HP)  # 16 bytes
        with pytest.raises(smat.SmatError):
            plan.adamw_fused_dev(state, torch.zeros(3, dtype=torch.int32, device=DEV)[1:3], cfg.lam, HP)  # misaligned
        with pytest.raises(smat.SmatError):
            plan.grad_norm_dev(state, cfg.lam)                                    # no output
        with pytest.raises(smat.SmatError):
            plan.grad_norm_dev(state, cfg.lam, max_norm=0.0, clip_coef=torch.zeros(1, device=DEV))
        plan.grad_norm_dev(state, cfg.lam, sumsq=sq)
        plan.simulate_dev(state)
        plan.switch_storage(smat.SMAT_SIMULATED)
        with pytest.raises(smat.SmatError):
            plan.adamw_fused_dev(state, adam, cfg.lam, HP)                      # simulated storage active
        plan.switch_storage(smat.SMAT_EXPERT)
        plan.adamw_fused_dev(state, adam.tensor, cfg.lam, HP)                   # a plain 8-byte tensor
        torch.cuda.synchronize()
    assert sq.item() > 0


def test_uploads_refused_under_capture(mini):
    """Calls that upload host tables through staging refuse to be captured; the capture itself stays
    usable and replays the device-driven call recorded before the refusal."""
    cfg, inp = mini
    th, t0, gs = list_tensors(inp)
    out_d, gt = fresh(inp)
    out_e, _ = fresh(inp)
    base = base_params(cfg, inp, 4)
    state = smat.StepState(cfg.smat_seed, 4, 0.625)
    refused = []
    with smat.Plan(th, out_d, t0, gs, gt) as pd, smat.Plan(th, out_e, t0, gs, gt) as pe:
        pd.set_params(base)
        pe.set_params(base)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            pd.simulate_dev(state)
            for call in (lambda: pd.set_params(base), lambda: pd.set_grads(grad_sims=gs),
                         lambda: pd.bind_adam_state([torch.empty_like(x) for x in th], [torch.empty_like(x) for x in th])):
                try:
                    call()
                except smat.SmatError as e:
                    refused.append(str(e))
        graph.replay()
        pe.simulate_dev(state)
        torch.cuda.synchronize()
        del graph
    assert len(refused) == 3 and all("cannot be captured" in m for m in refused), refused
    assert same_bits(out_d, out_e)


# ---------------------------------------------------------------- the step's scale drawn on the device
@pytest.mark.parametrize("seed,step0,alpha_min", [(0, 0, 0.2), (2 ** 64 - 1, 41, 0.1), (12345, 2 ** 30 - 5, 0.75),
                                                  (7, 100, 0.0), (7, 100, 1.0), (9, 2 ** 30 - 2, 0.3)])
def test_step_advance_matches_oracle(seed, step0, alpha_min):
    st = smat.StepState(seed, step0, -1.0)
    st.advance(alpha_min, 0)                     # the scale of the current step
    torch.cuda.synchronize()
    assert st.step_view.item() == step0
    assert st.scale_view.item() == oracle.scale_draw(seed, step0, alpha_min)
    for k in range(1, 4):
        st.advance(alpha_min)
        torch.cuda.synchronize()
        step = (step0 + k) % 2 ** 30             # steps live in [0, 2^30): past the last one, step 0 again
        assert st.step_view.item() == step
        assert st.scale_view.item() == oracle.scale_draw(seed, step, alpha_min)
    assert st.seed_view.item() == (seed if seed < 2 ** 63 else seed - 2 ** 64)
    with pytest.raises(smat.SmatError):
        st.advance(1.5)


def test_graph_with_scale_drawn_on_the_device(mini):
    """One graph: advance (step + 1, scale of that step), simulate, backward; each replay equals the
    host-driven step with the oracle's scale for that step."""
    cfg, inp = mini
    th, t0, gs = list_tensors(inp)
    out_d, gt_d = fresh(inp)
    out_h, gt_h = fresh(inp)
    base = base_params(cfg, inp, 0)
    step0, amin = 60, 0.2
    state = smat.StepState(cfg.smat_seed, step0, 1.0)
    with smat.Plan(th, out_d, t0, gs, gt_d) as pd, smat.Plan(th, out_h, t0, gs, gt_h) as ph:
        pd.set_params(base)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            state.advance(amin)
            pd.simulate_dev(state)
            pd.backward_dev(state, cfg.lam, False)
        for k in range(1, 4):
            for o in out_d:
                o.fill_(float("nan"))
            graph.replay()
            step = step0 + k
            scale = oracle.scale_draw(cfg.smat_seed, step, amin)
            ph.set_params(scaled(base, scale))
            ph.simulate(cfg.smat_seed, step)
            ph.backward(cfg.smat_seed, step, cfg.lam, False)
            torch.cuda.synchronize()
            assert state.step_view.item() == step and state.scale_view.item() == scale
            assert same_bits(out_d, out_h), k
            assert same_bits(gt_d, gt_h), k
        del graph


# ---------------------------------------------------------------- a whole captured training step
def _mlp(seed):
    g = torch.Generator().manual_seed(seed)
    model = torch.nn.Sequential(torch.nn.Linear(32, 96), torch.nn.GELU(), torch.nn.Linear(96, 24))
    with torch.no_grad():
        for p in model.parameters():
            p.copy_(torch.randn(p.shape, generator=g) * 0.1)
    return model.to(DEV)


def test_captured_training_step_with_a_model():
    """A simulated training step captured once with the model inside: advance (step + 1, its
    scale), simulate into the buffers the model reads, forward and backward into static gradient
    tensors, gradient norm and clipped fused AdamW on the expert storage, the optimizer's step count
    advanced on the device.  Three replays against the same steps run eagerly through the
    host-driven calls on a twin model."""
    x = torch.randn(64, 32, generator=torch.Generator().manual_seed(1)).to(DEV)
    y = torch.randn(64, 24, generator=torch.Generator().manual_seed(2)).to(DEV)
    seed, step0, amin, lam, lr, k0, max_norm = 99, 10, 0.2, 1.0, 1e-3, 0, 0.05
    hp = dict(beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, grad_scale=1.0)
    keeps = [0.5, 1.0, 0.5, 1.0]                        # weights masked, biases not
    twins = []
    for _ in range(2):
        model = _mlp(7)
        params = list(model.parameters())
        master = [p.data for p in params]
        theta0 = [(p.data + 0.01 * torch.randn(p.shape, generator=torch.Generator().manual_seed(3)).to(DEV))
                  for p in params]
        buffers = [torch.empty_like(p) for p in params]
        for p, b in zip(params, buffers):
            p.data = b                                  # the model reads theta~ from here on
            p.grad = torch.zeros_like(b)                # static gradient tensors at theta~
        m1 = [torch.zeros_like(m) for m in master]
        m2 = [torch.zeros_like(m) for m in master]
        plan = smat.Plan(master, buffers, theta0, [p.grad for p in params])
        plan.set_params(smat.op_params_array(len(params), 1.0, keeps, 1e-3, 1, smat.SMAT_NOISE_UNIFORM))
        plan.bind_adam_state(m1, m2)
        twins.append((model, params, master, plan, m1, m2))

    def loss_backward(model, params):
        for p in params:
            p.grad.zero_()
        torch.nn.functional.mse_loss(model(x), y).backward()

    # A: device-driven, then captured
    model_a, params_a, master_a, plan_a, m1_a, m2_a = twins[0]
    state, adam = smat.StepState(seed, step0, 1.0), smat.AdamStepState(lr, k0)
    coef_a = torch.zeros(1, device=DEV)

    def step_a():
        state.advance(amin)
        adam.step_view.add_(1)
        plan_a.simulate_dev(state)
        loss_backward(model_a, params_a)
        plan_a.grad_norm_dev(state, lam, False, max_norm, clip_coef=coef_a)
        plan_a.adamw_fused_dev(state, adam, lam, hp, False, coef_a)

    # B: the same steps issued from the host
    model_b, params_b, master_b, plan_b, m1_b, m2_b = twins[1]
    coef_b = torch.zeros(1, device=DEV)
    base = smat.op_params_array(len(params_b), 1.0, keeps, 1e-3, 1, smat.SMAT_NOISE_UNIFORM)

    def step_b(step, k):
        arr = base.copy()
        arr["s"] = smat.scale_draw(seed, step, amin)
        plan_b.set_params(arr)
        plan_b.simulate(seed, step)
        loss_backward(model_b, params_b)
        plan_b.grad_norm(seed, step, lam, False, max_norm, clip_coef=coef_b)
        plan_b.adamw_fused(seed, step, lam, dict(hp, lr=lr, step=k), False, coef_b)

    def same_state():
        torch.cuda.synchronize()
        for a, b in zip(master_a + m1_a + m2_a, master_b + m1_b + m2_b):
            torch.testing.assert_close(a, b, rtol=1e-6, atol=1e-9)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                       # eager warmup steps before the capture
        for _ in range(2):
            step_a()
    torch.cuda.current_stream().wait_stream(side)
    for r in (1, 2):
        step_b(step0 + r, k0 + r)
    same_state()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step_a()
    for r in range(3, 6):
        graph.replay()
        step_b(step0 + r, k0 + r)
        same_state()
        assert 0 < coef_a.item() <= 1 and state.step_view.item() == step0 + r
    assert coef_a.item() < 1                            # the clipping is active
    del graph
    for t in twins:
        t[3].close()


def test_device_calls_on_empty_lists_and_tensors():
    """An empty plan and zero-size tensors in a list: the device-driven calls launch nothing for them
    and leave every other tensor as the host-driven calls do."""
    state, adam = smat.StepState(3, 4, 0.5), smat.AdamStepState(1e-3, 2)
    sq = torch.full((1,), 7.0, dtype=torch.float64, device=DEV)
    with smat.Plan([], [], [], [], []) as plan:
        plan.set_params([])
        plan.bind_adam_state([], [])
        plan.simulate_dev(state)
        plan.backward_dev(state, 1.0)
        plan.grad_norm_dev(state, 1.0, sumsq=sq)
        plan.adamw_fused_dev(state, adam, 1.0, dict(beta1=0.9, beta2=0.99, eps=1e-8, weight_decay=0.0))
        torch.cuda.synchronize()
    assert sq.item() == 0.0
    g = torch.Generator(DEV).manual_seed(9)
    sizes = [0, 37, 0, 4100]
    res = {}
    for mode in ("dev", "host"):
        th = [torch.randn(n, device=DEV, generator=torch.Generator(DEV).manual_seed(n + 1)) for n in sizes]
        t0 = [x.to(torch.bfloat16) for x in th]
        gs = [(torch.randn(n, device=DEV, generator=g) * 0.0 + 0.01 * (i + 1)).to(torch.bfloat16)
              for i, n in enumerate(sizes)]
        gt = [torch.zeros(n, device=DEV) for n in sizes]
        out = [torch.full((n,), float("nan"), device=DEV, dtype=torch.bfloat16) for n in sizes]
        base = [dict(s=0.5 + 0.1 * i, keep=0.6, sigma=1e-3, rescale=1) for i in range(len(sizes))]
        with smat.Plan(th, out, t0, gs, gt) as plan:
            if mode == "dev":
                plan.set_params(base)
                plan.simulate_dev(state)
                plan.backward_dev(state, 0.5, True)
            else:
                plan.set_params(scaled(base, 0.5))
                plan.simulate(3, 4)
                plan.backward(3, 4, 0.5, True)
            torch.cuda.synchronize()
        res[mode] = (out, gt)
    assert same_bits(res["dev"][0], res["host"][0]) and same_bits(res["dev"][1], res["host"][1])


def test_rejected_records_name_their_tensor(mini):
    cfg, inp = mini
    th, t0, gs = list_tensors(inp)
    out, gt = fresh(inp)
    bad = base_params(cfg, inp, 1)
    bad[4] = dict(bad[4], keep=1.5)
    with smat.Plan(th, out, t0, gs, gt) as plan:
        with pytest.raises(smat.SmatError, match="smat_plan_set_params: tensor 4: keep"):
            plan.set_params(bad)
        with pytest.raises(smat.SmatError, match="smat_plan_set_grads: tensor 2"):
            plan.set_grads(grad_thetas=[x if i != 2 else th[2] for i, x in enumerate(gt)])   # over theta
    t0s = [t.to(torch.bfloat16) for t in th[:3]]
    outs = [torch.empty_like(t) for t in t0s]
    experts = [[t.clone() for t in t0s] for _ in range(3)]
    with smat.MergePlan(t0s, outs, experts) as m:
        terms = [[dict(gamma=0.3, keep=1.0, seed=j) for j in range(3)] for _ in range(3)]
        terms[1][2] = dict(gamma=0.3, keep=-1.0, seed=2)
        with pytest.raises(smat.SmatError, match="smat_merge_multi: tensor 1, expert 2"):
            m.merge(terms)
    torch.cuda.synchronize()
