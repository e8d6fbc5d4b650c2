"""Seeded random sweeps of the simulate/backward, the fused AdamW step and the merge against the
oracle, over combinations the hand-written cases do not enumerate: sizes from 1 to ~70K, buffer
misalignment, element offsets anywhere below 2^40 (and tiles that cross a multiple of 2^34), all
dtype mixes, keep at 0, tiny, just below 1 and 1, negative and zero scales, every noise form,
rescale on and off, accumulate and overwrite, random optimizer settings, 1-16 experts.  Single
tensors through the single-tensor entry points, ragged lists through a plan."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_33437_amd as smat
from helpers import host
from tolerances import check_grad, check_theta_tilde, nonstrict_within_cap, ordered, theta_tilde_report

pytestmark = pytest.mark.gpu
DEV = "cuda"
DT = {"bf16": torch.bfloat16, "f32": torch.float32}
KEEP_FP32_BELOW_1 = float(np.nextafter(np.float32(1.0), np.float32(0.0)))


def draw_case(rng):
    n = int(np.exp(rng.uniform(0.0, np.log(70000.0))))
    off = int(rng.choice([0, 4 * int(rng.integers(0, 2 ** 38)), int(rng.integers(0, 2 ** 40)),
                          2 ** 34 - 4 * int(rng.integers(1, 600)), 2 ** 35 - int(rng.integers(1, 3000))]))
    keep = float(np.float32(rng.choice([0.0, 1.0, 0.5, rng.uniform(0.01, 0.99), 1e-9, KEEP_FP32_BELOW_1])))
    s = float(np.float32(rng.choice([0.0, 1.0, rng.uniform(-1.0, 2.0)])))
    sigma = float(np.float32(rng.choice([0.0, 10 ** rng.uniform(-4, -2)])))
    p = dict(s=s, keep=keep, sigma=sigma, rescale=int(rng.integers(0, 2)), noise_kind=int(rng.integers(0, 3)))
    return n, off, p, int(rng.integers(0, 4))


def tensors(rng, n, shift, t0_dt, out_dt, g_dt, gen):
    base = torch.randn(n + 8, device=DEV, generator=gen) * 0.02
    th = base[shift:shift + n]
    t0 = (base + torch.randn(n + 8, device=DEV, generator=gen) * 1e-3).to(DT[t0_dt])[shift:shift + n]
    out = torch.empty(n + 8, dtype=DT[out_dt], device=DEV)[shift:shift + n]
    gs = (torch.randn(n + 8, device=DEV, generator=gen) * 1e-2).to(DT[g_dt])[shift:shift + n]
    gt = (torch.randn(n + 8, device=DEV, generator=gen) * 1e-3)[shift:shift + n]
    return th, t0, out, gs, gt


def check_sim(th, t0, out, p, seed, step, tid, off, what):
    thn, _ = host(th)
    t0n, t0_dt = host(t0)
    got, out_dt = host(out)
    y, kept, eps = oracle.simulate_f64(thn, t0n, t0_dt, p, seed, step, tid, off)
    coef = np.where(kept, oracle.coefficient(p["s"], p["keep"], p["rescale"]), 0.0)
    ok, strict = check_theta_tilde(got, out_dt, y, thn, oracle.as_f64(t0n, t0_dt), coef, eps, p["sigma"])
    assert ok.all(), f"{what}: {np.count_nonzero(~ok)} theta~ mismatches, first {np.flatnonzero(~ok)[:5]}"
    if out_dt == "bf16":
        n, loose, _, worst_strict = theta_tilde_report(got, oracle.round_to_bf16_bits(y), strict)
        assert worst_strict <= 1, what
        assert nonstrict_within_cap(loose, n), (what, loose, n)
    return kept


def check_bwd(got, gs, g_old, p, lam, seed, step, tid, off, kept, what):
    gsn, gs_dt = host(gs)
    want = oracle.backward_accum(gsn, gs_dt, g_old, p, lam, seed, step, tid, off)
    incr = np.abs(oracle.simulated_gradient(gsn, gs_dt, p, lam, seed, step, tid, off))
    assert check_grad(got, want, g_old, incr).all(), what
    np.testing.assert_array_equal(got.view(np.uint32)[~kept], g_old.view(np.uint32)[~kept], err_msg=what)


def test_random_single_tensors():
    rng = np.random.default_rng(20260)
    gen = torch.Generator(DEV).manual_seed(20260)
    for case in range(120):
        n, off, p, shift = draw_case(rng)
        t0_dt, out_dt, g_dt = (str(rng.choice(["bf16", "f32"])) for _ in range(3))
        seed, step, tid = int(rng.integers(0, 2 ** 63)), int(rng.integers(0, 2 ** 30)), int(rng.integers(0, 2 ** 32))
        lam = float(np.float32(rng.uniform(-1.0, 2.0)))
        what = f"case {case}: n={n} off={off} shift={shift} dtypes={t0_dt}/{out_dt}/{g_dt} p={p} lam={lam}"
        th, t0, out, gs, gt = tensors(rng, n, shift, t0_dt, out_dt, g_dt, gen)
        g_old = host(gt)[0]
        smat.smat_simulate(th, t0, out, p, seed, step, tid, off)
        smat.smat_backward_accum(gs, gt, p, lam, seed, step, tid, off)
        torch.cuda.synchronize()
        kept = check_sim(th, t0, out, p, seed, step, tid, off, what)
        check_bwd(host(gt)[0], gs, g_old, p, lam, seed, step, tid, off, kept, what)


def test_random_lists():
    rng = np.random.default_rng(20261)
    gen = torch.Generator(DEV).manual_seed(20261)
    for case in range(50):
        count = int(rng.integers(1, 7))
        t0_dt, out_dt, g_dt = (str(rng.choice(["bf16", "f32"])) for _ in range(3))
        seed, step = int(rng.integers(0, 2 ** 63)), int(rng.integers(0, 2 ** 30))
        lam = float(np.float32(rng.uniform(-1.0, 2.0)))
        items = [draw_case(rng) for _ in range(count)]
        ids = [int(x) for x in rng.choice(2 ** 32, size=count, replace=False)]
        ts = [tensors(rng, n, shift, t0_dt, out_dt, g_dt, gen) for n, _, _, shift in items]
        th, t0, out, gs, gt = (list(x) for x in zip(*ts))
        fresh = [torch.full_like(g, float("nan")) for g in gt]
        offs, params = [it[1] for it in items], [it[2] for it in items]
        g_old = [host(g)[0] for g in gt]
        with smat.Plan(th, out, t0, gs, gt, tensor_ids=ids, elem_offsets=offs) as plan:
            plan.set_params(params)
            plan.simulate(seed, step)
            plan.backward(seed, step, lam, accumulate=True)
            plan.set_grads(None, fresh)
            plan.backward(seed, step, lam, accumulate=False)
            torch.cuda.synchronize()
        for i in range(count):
            n, off, p, shift = items[i]
            what = f"list {case} tensor {i}: n={n} off={off} shift={shift} dtypes={t0_dt}/{out_dt}/{g_dt} p={p}"
            kept = check_sim(th[i], t0[i], out[i], p, seed, step, ids[i], off, what)
            check_bwd(host(gt[i])[0], gs[i], g_old[i], p, lam, seed, step, ids[i], off, kept, what)
            zero = np.zeros(n, np.float32)
            check_bwd(host(fresh[i])[0], gs[i], zero, p, lam, seed, step, ids[i], off, kept, what + " (overwrite)")


def draw_adam(rng):
    return dict(lr=float(10 ** rng.uniform(-6, -2)), beta1=float(rng.choice([0.0, 0.9, rng.uniform(0.5, 0.99)])),
                beta2=float(rng.choice([0.999, rng.uniform(0.9, 0.9999)])), eps=float(10 ** rng.uniform(-10, -6)),
                weight_decay=float(rng.choice([0.0, 1e-3, rng.uniform(0.0, 0.1)])),
                grad_scale=float(rng.choice([1.0, rng.uniform(0.1, 2.0)])), step=int(rng.integers(1, 1000)))


def check_adamw(th, m1, m2, old, gs, p, lam, hp, seed, step, tid, off, acc, what):
    from tolerances import check_adam
    gsn, gs_dt = host(gs)
    _, f64 = oracle.adamw_fused(gsn, gs_dt, old[0], old[1], old[2], p, lam, hp, seed, step, tid, off, grad_acc=acc)
    gmag = np.abs(oracle.simulated_gradient(gsn, gs_dt, p, lam, seed, step, tid, off, None, hp["grad_scale"]))
    if acc is not None:
        gmag = gmag + abs(float(np.float32(hp["grad_scale"]))) * np.abs(np.asarray(acc, dtype=np.float64))
    ok = check_adam((host(th)[0], host(m1)[0], host(m2)[0]), old, f64, hp, gmag)
    for name, o in zip(("theta", "exp_avg", "exp_avg_sq"), ok):
        assert o.all(), f"{what}: {name} {np.count_nonzero(~o)} mismatches, first {np.flatnonzero(~o)[:5]}"


def test_random_fused_adamw():
    rng = np.random.default_rng(20262)
    gen = torch.Generator(DEV).manual_seed(20262)
    for case in range(40):
        n, off, p, shift = draw_case(rng)
        g_dt = str(rng.choice(["bf16", "f32"]))
        accumulate = bool(rng.integers(0, 2))
        seed, step, tid = int(rng.integers(0, 2 ** 63)), int(rng.integers(0, 2 ** 30)), int(rng.integers(0, 2 ** 32))
        lam = float(np.float32(rng.uniform(-1.0, 2.0)))
        hp = draw_adam(rng)
        what = f"case {case}: n={n} off={off} shift={shift} g={g_dt} acc={accumulate} p={p} lam={lam} hp={hp}"
        th = (torch.randn(n + 8, device=DEV, generator=gen) * 0.02)[shift:shift + n]
        m1 = (torch.randn(n + 8, device=DEV, generator=gen) * 1e-3)[shift:shift + n]
        m2 = (torch.rand(n + 8, device=DEV, generator=gen) * 1e-6)[shift:shift + n]
        gs = (torch.randn(n + 8, device=DEV, generator=gen) * 1e-2).to(DT[g_dt])[shift:shift + n]
        acc = (torch.randn(n + 8, device=DEV, generator=gen) * 1e-3)[shift:shift + n] if accumulate else None
        old = (host(th)[0], host(m1)[0], host(m2)[0])
        accn = host(acc)[0] if accumulate else None
        smat.smat_adamw_fused(gs, th, m1, m2, p, lam, hp, seed, step, tid, off, grad_acc=acc)
        torch.cuda.synchronize()
        check_adamw(th, m1, m2, old, gs, p, lam, hp, seed, step, tid, off, accn, what)


def test_random_merges():
    from tolerances import check_merge
    rng = np.random.default_rng(20263)
    gen = torch.Generator(DEV).manual_seed(20263)
    for case in range(40):
        n, off, _, shift = draw_case(rng)
        nexp = int(rng.integers(1, 17))
        e_dt, t0_dt, out_dt = (str(rng.choice(["bf16", "f32"])) for _ in range(3))
        tid = int(rng.integers(0, 2 ** 32))
        terms = [dict(gamma=float(np.float32(rng.uniform(-1.0, 1.5))),
                      keep=float(np.float32(rng.choice([0.0, 1.0, rng.uniform(0.05, 0.99), KEEP_FP32_BELOW_1]))),
                      rescale=int(rng.integers(0, 2)), seed=int(rng.integers(0, 2 ** 63)),
                      step=int(rng.integers(0, 2 ** 30))) for _ in range(nexp)]
        what = f"case {case}: n={n} off={off} shift={shift} nexp={nexp} dtypes={e_dt}/{t0_dt}/{out_dt}"
        base = torch.randn(n + 8, device=DEV, generator=gen) * 0.02
        t0 = base.to(DT[t0_dt])[shift:shift + n]
        ex = [(base + torch.randn(n + 8, device=DEV, generator=gen) * 1e-3).to(DT[e_dt])[shift:shift + n]
              for _ in range(nexp)]
        out = torch.empty(n + 8, dtype=DT[out_dt], device=DEV)[shift:shift + n]
        smat.smat_merge(ex, t0, out, terms, tid, off)
        torch.cuda.synchronize()
        exn = [host(x) for x in ex]
        t0n, t0dt = host(t0)
        y = oracle.merge_f64([x for x, _ in exn], e_dt, t0n, t0dt, terms, tid, off)
        b = oracle.as_f64(t0n, t0dt)
        A, used = np.abs(b).copy(), 0
        for (x, dt), t in zip(exn, terms):
            kept = oracle.keep_mask(t["seed"], t["step"], tid, off, n, t["keep"])
            tj = oracle.coefficient(t["gamma"], t["keep"], t["rescale"])
            A += np.where(kept, abs(tj) * (np.abs(oracle.as_f64(x, dt)) + np.abs(b)), 0.0)
            used += float(np.float32(t["keep"])) > 0
        got, _ = host(out)
        ok, strict = check_merge(got, out_dt, y, A, max(used, 1))
        assert ok.all(), f"{what}: {np.count_nonzero(~ok)} mismatches, first {np.flatnonzero(~ok)[:5]}"
        if out_dt == "bf16":
            assert np.abs(ordered(got) - ordered(oracle.round_to_bf16_bits(y)))[strict].max(initial=0) <= 1, what


def test_random_list_norms():
    from tolerances import SQNORM_ULPS, U, check_sqnorm
    rng = np.random.default_rng(20264)
    gen = torch.Generator(DEV).manual_seed(20264)
    for case in range(30):
        count = int(rng.integers(1, 7))
        g_dt = str(rng.choice(["bf16", "f32"]))
        accumulate = bool(rng.integers(0, 2))
        seed, step = int(rng.integers(0, 2 ** 63)), int(rng.integers(0, 2 ** 30))
        lam = float(np.float32(rng.uniform(-1.0, 2.0)))
        items = [draw_case(rng) for _ in range(count)]
        ids = [int(x) for x in rng.choice(2 ** 32, size=count, replace=False)]
        ts = [tensors(rng, n, shift, "bf16", "bf16", g_dt, gen) for n, _, _, shift in items]
        th, t0, out, gs, gt = (list(x) for x in zip(*ts))
        offs, params = [it[1] for it in items], [it[2] for it in items]
        what = f"list {case}: sizes={[it[0] for it in items]} offs={offs} g={g_dt} acc={accumulate} lam={lam}"
        want, m2 = 0.0, 0.0
        for i in range(count):
            gsn, gs_dt = host(gs[i])
            acc = host(gt[i])[0] if accumulate else None
            want += oracle.grad_sqnorm(gsn, gs_dt, params[i], lam, seed, step, ids[i], offs[i], acc)
            m = np.abs(oracle.simulated_gradient(gsn, gs_dt, params[i], lam, seed, step, ids[i], offs[i]))
            if acc is not None:
                m = m + np.abs(acc.astype(np.float64))
            m2 += float(np.dot(m, m))
        sumsq = torch.zeros(1, dtype=torch.float64, device=DEV)
        coef = torch.zeros(1, dtype=torch.float32, device=DEV)
        max_norm = float(rng.uniform(0.1, 2.0)) * max(want, 1e-30) ** 0.5
        with smat.Plan(th, out, t0, gs, gt, tensor_ids=ids, elem_offsets=offs) as plan:
            plan.set_params(params)
            plan.grad_norm(seed, step, lam, accumulate, max_norm, sumsq, coef)
            torch.cuda.synchronize()
        assert check_sqnorm(sumsq.item(), want, m2), (what, sumsq.item(), want)
        if want > 0:
            want_coef = oracle.clip_coefficient(want ** 0.5, max_norm)
            rel = 0.5 * SQNORM_ULPS * U * m2 / want + 2 * U
            assert abs(coef.item() - want_coef) <= rel * want_coef + 2 * U, (what, coef.item(), want_coef)
