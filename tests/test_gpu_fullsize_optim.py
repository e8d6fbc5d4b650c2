"""Full-size parity of the optimizer side and of the N-expert merge on the 7B-shaped list, launched
as the benchmark launches them (one plan, one launch per operation over the whole list):

* the gradient-norm pass: checked against an fp64 torch reduction of the kept squares, the kept
  coordinates coming from smat_debug_draws (itself bit-exact against the oracle);
* the clipped fused AdamW step: sampled windows of every tensor against the oracle fed with the
  clipping factor the GPU used;
* the DARE + Task Arithmetic merge of seven bf16 experts: sampled windows against the oracle."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_33437_amd as smat
import workloads
from helpers import host
from tolerances import SQNORM_ULPS, U, check_adam, check_merge, ordered

pytestmark = pytest.mark.gpu
DEV = "cuda"
W = 256
HP = dict(lr=2e-5, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-3, grad_scale=1.0, step=7)


def windows(n, rng):
    if n <= 4 * W:
        return [(0, n)]
    r = int(rng.integers(W, n - 2 * W))
    return [(0, W), (r, r + W), (n - W - 3, n)]


def test_fullsize_norm_and_clipped_fused_adamw_c4():
    torch.cuda.empty_cache()
    cfg = workloads.config("c4")
    print(f"[c4] generating {cfg.count} tensors, {cfg.numel} params and moments", flush=True)
    inp = workloads.make_inputs(cfg, device=DEV)
    outs = [torch.empty(t.numel(), dtype=torch.bfloat16, device=DEV) for t in inp.theta]
    g = torch.Generator(DEV).manual_seed(5)
    m1 = [torch.randn(t.numel(), device=DEV, generator=g) * 1e-3 for t in inp.theta]
    m2 = [torch.rand(t.numel(), device=DEV, generator=g) * 1e-6 for t in inp.theta]
    step = 7
    params = workloads.step_params(cfg, inp.settings, step)
    rng = np.random.default_rng(41)
    wins = [windows(t.numel(), rng) for t in inp.theta]
    samples = [[(a, b, host(inp.theta[i].view(-1)[a:b])[0], host(m1[i][a:b])[0], host(m2[i][a:b])[0],
                 host(inp.grad_sim[i].view(-1)[a:b])[0]) for a, b in ws] for i, ws in enumerate(wins)]
    # reference squared norm: fp64 sum of the kept squares, the mask from the debug draws
    ref = 0.0
    for i, p in enumerate(params):
        gs = inp.grad_sim[i].view(-1).double()
        if p["keep"] < 1.0:
            kept = torch.empty(gs.numel(), dtype=torch.uint8, device=DEV)
            smat.smat_debug_draws(gs.numel(), p, cfg.smat_seed, step, i, 0, kept=kept)
            gs = gs * kept.double()
            del kept
        c = cfg.lam * oracle.coefficient(p["s"], p["keep"], p["rescale"])
        ref += c * c * float((gs * gs).sum())
        del gs
    sumsq = torch.zeros(1, dtype=torch.float64, device=DEV)
    coef = torch.zeros(1, dtype=torch.float32, device=DEV)
    max_norm = 0.5 * math.sqrt(ref)
    with smat.Plan(inp.theta, outs, inp.theta0, inp.grad_sim, inp.grad_theta) as plan:
        plan.set_params(params)
        plan.bind_adam_state(m1, m2)
        plan.grad_norm(cfg.smat_seed, step, cfg.lam, False, max_norm, sumsq, coef)
        plan.adamw_fused(cfg.smat_seed, step, cfg.lam, HP, grad_scale_dev=coef)
        torch.cuda.synchronize()
    got = float(sumsq.item())
    print(f"[c4] sumsq gpu {got:.9e} reference {ref:.9e}", flush=True)
    assert abs(got - ref) <= SQNORM_ULPS * U * ref
    c = float(coef.item())
    assert abs(c - oracle.clip_coefficient(math.sqrt(ref), max_norm)) <= (0.5 * SQNORM_ULPS + 2) * U * c
    hp = dict(HP, grad_scale=c)
    for i, ws in enumerate(samples):
        for a, b, th, a1, a2, gsn in ws:
            _, f64 = oracle.adamw_fused(gsn, "bf16", th, a1, a2, params[i], cfg.lam, hp, cfg.smat_seed, step, i, a)
            gmag = c * np.abs(oracle.simulated_gradient(gsn, "bf16", params[i], cfg.lam, cfg.smat_seed, step, i, a))
            got3 = (host(inp.theta[i].view(-1)[a:b])[0], host(m1[i][a:b])[0], host(m2[i][a:b])[0])
            for name, ok in zip(("theta", "exp_avg", "exp_avg_sq"), check_adam(got3, (th, a1, a2), f64, hp, gmag)):
                assert ok.all(), f"tensor {i} [{a},{b}) {name}: {np.count_nonzero(~ok)} mismatches"
    del inp, outs, m1, m2
    torch.cuda.empty_cache()


def test_fullsize_dare_merge_c4():
    torch.cuda.empty_cache()
    cfg = workloads.config("c4")
    N = 7
    print(f"[c4] generating {N} experts of {cfg.numel} params", flush=True)
    t0s, experts = workloads.make_experts(cfg, N, device=DEV)
    outs = [torch.empty_like(t) for t in t0s]
    masked = [spec.kind == "linear" for spec in cfg.specs]
    terms = [[dict(gamma=0.3, keep=0.7 if m else 1.0, seed=0xDA4E + j, step=0) for j in range(N)] for m in masked]
    with smat.MergePlan(t0s, outs, experts) as plan:
        plan.merge(terms)
        torch.cuda.synchronize()
    rng = np.random.default_rng(43)
    worst = 0
    for i in range(cfg.count):
        n = t0s[i].numel()
        for a, b in windows(n, rng):
            t0 = host(t0s[i].view(-1)[a:b])[0]
            xs = [host(e[i].view(-1)[a:b])[0] for e in experts]
            y = oracle.merge_f64(xs, "bf16", t0, "bf16", terms[i], i, a)
            b0 = oracle.as_f64(t0, "bf16")
            A = np.abs(b0).copy()
            for x, t in zip(xs, terms[i]):
                kept = oracle.keep_mask(t["seed"], t["step"], i, a, b - a, t["keep"])
                A += np.where(kept, oracle.coefficient(t["gamma"], t["keep"], 1) * (np.abs(oracle.as_f64(x, "bf16"))
                                                                                    + np.abs(b0)), 0.0)
            got = host(outs[i].view(-1)[a:b])[0]
            ok, strict = check_merge(got, "bf16", y, A, N)
            assert ok.all(), f"tensor {i} [{a},{b}): {np.count_nonzero(~ok)} merge mismatches"
            worst = max(worst, int(np.abs(ordered(got) - ordered(oracle.round_to_bf16_bits(y)))[strict].max(initial=0)))
    assert worst <= 1
    del t0s, experts, outs
    torch.cuda.empty_cache()
