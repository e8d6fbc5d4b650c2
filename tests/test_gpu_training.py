"""GPU parity of the training-loop wrapper (paper_2609_33437_amd.training) on a small synthetic
decoder.  Checked against the oracle:

* theta~ seen by the model on a simulated step;
* the expert gradient lam alpha m (.) g~ left for the optimizer;
* the fused Adam/AdamW update driven by the torch optimizer's own state.

Also checked: the schedule leaves ordinary steps untouched; the forward and backward really run on
the buffers; offload mode reproduces resident mode bit for bit across cycles; a bf16 autocast loop
runs end to end."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_33437_amd as smat
from paper_2609_33437_amd.training import SimulatedMergeTraining
from helpers import host
from tolerances import SQNORM_ULPS, U, check_adam, check_grad, check_sqnorm, check_theta_tilde, ordered
from workloads.model import TINY, make_decoder, token_batches

pytestmark = pytest.mark.gpu
DEV = "cuda"
SEED = 0x51A7


def base_weights(model, seed=3, scale=0.01):
    """theta0: the model's weights moved by a seeded displacement, so that Delta != 0."""
    g = torch.Generator().manual_seed(seed)
    return {n: (p.detach().cpu() + scale * torch.randn(p.shape, generator=g)).to(DEV)
            for n, p in model.named_parameters()}


def wrap(model, **kw):
    kw.setdefault("buffer_dtype", torch.float32)
    return SimulatedMergeTraining.from_module(model, keep=0.5, alpha_min=0.2, sigma=2e-3,
                                              theta0=base_weights(model), seed=SEED, **kw)


def op(w, i):
    return dict(s=w.alpha, keep=w.keep[i], sigma=w.sigma[i], rescale=w.rescale, noise_kind=w.noise_kind)


def check_simulated(w, masters, step):
    for i, (p, m) in enumerate(zip(w.params, masters)):
        th, _ = host(m)
        t0, t0_dt = host(w.theta0[i] if not w.offload else w.theta0_host[i])
        y, kept, eps = oracle.simulate_f64(th, t0, t0_dt, op(w, i), SEED, step, i)
        coef = np.where(kept, oracle.coefficient(w.alpha, w.keep[i], w.rescale), 0.0)
        got, out_dt = host(p.data)
        ok, strict = check_theta_tilde(got, out_dt, y, th, oracle.as_f64(t0, t0_dt), coef, eps, w.sigma[i])
        assert ok.all(), f"{w.names[i]}: {np.count_nonzero(~ok)} theta~ mismatches"
        if out_dt == "bf16":
            assert np.abs(ordered(got) - ordered(oracle.round_to_bf16_bits(y)))[strict].max(initial=0) <= 1


def test_simulated_step_matches_oracle():
    torch.manual_seed(0)
    model = make_decoder(TINY, 5, DEV)
    tokens = token_batches(TINY, 2, 24, 1, 7, DEV)[0]
    w = wrap(model)
    masters = [p.detach().clone() for p in w.params]
    ids = [p.data_ptr() for p in w.params]
    for step in range(3):                               # ordinary steps touch nothing
        assert not w.begin(step) and not w.active
        assert [p.data_ptr() for p in w.params] == ids
    assert w.begin(3) and w.active
    assert 0.2 <= w.alpha <= 1.0
    assert w.alpha == oracle.scale_draw(SEED, 3, 0.2)    # a function of (seed, step): resumable
    assert all(p.data_ptr() == b.data_ptr() for p, b in zip(w.params, w.buffers))
    check_simulated(w, masters, 3)
    # the forward and backward run on theta~: compare with a copy of the model holding theta~
    ref = make_decoder(TINY, 5, DEV)
    with torch.no_grad():
        for q, p in zip(ref.parameters(), w.params):
            q.copy_(p.data)
    loss = model.loss(tokens)
    loss.backward()
    ref_loss = ref.loss(tokens)
    ref_loss.backward()
    assert torch.allclose(loss, ref_loss, rtol=1e-6, atol=0)
    for p, q in zip(w.params, ref.parameters()):
        torch.testing.assert_close(p.grad, q.grad, rtol=1e-5, atol=1e-7)
    g_sim = [host(p.grad)[0] for p in w.params]    # the gradients at theta~ autograd produced
    w.end()
    assert not w.active
    for i, (p, m) in enumerate(zip(w.params, masters)):
        assert p.data_ptr() == ids[i] and torch.equal(p.data, m)      # expert storage untouched
        zeros = np.zeros(p.numel(), np.float32)
        want = oracle.backward_accum(g_sim[i], "f32", zeros, op(w, i), w.lam, SEED, 3, i)
        incr = np.abs(oracle.simulated_gradient(g_sim[i], "f32", op(w, i), w.lam, SEED, 3, i))
        ok = check_grad(host(p.grad)[0], want, zeros, incr)
        assert ok.all(), f"{w.names[i]}: {np.count_nonzero(~ok)} gradient mismatches"
    w.close()


@pytest.mark.parametrize("torch_fused", [False, True])
def test_fused_adamw_step_matches_oracle(torch_fused):
    model = make_decoder(TINY, 9, DEV)
    batches = token_batches(TINY, 2, 16, 4, 11, DEV)
    w = wrap(model)
    opt = torch.optim.AdamW(w.params, lr=1e-3, betas=(0.9, 0.95), eps=1e-8, weight_decay=0.05, fused=torch_fused)
    for step in range(3):
        opt.zero_grad()
        assert not w.begin(step)
        model.loss(batches[step]).backward()
        opt.step()
    opt.zero_grad()
    assert w.begin(3)
    model.loss(batches[3]).backward()
    # p.data is theta~ here; the update applies to the expert storage
    old = [(host(m)[0], host(opt.state[p]["exp_avg"])[0], host(opt.state[p]["exp_avg_sq"])[0])
           for p, m in zip(w.params, w.master)]
    g_sim = [host(p.grad)[0] for p in w.params]    # the gradients at theta~ autograd produced
    ops = [op(w, i) for i in range(len(w.params))]
    w.end(opt, fused=True)
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.05, grad_scale=1.0, step=4)
    for i, p in enumerate(w.params):
        st = opt.state[p]
        assert int(float(st["step"])) == 4 and p.grad is None
        _, f64 = oracle.adamw_fused(g_sim[i], "f32", *old[i], ops[i], w.lam, hp, SEED, 3, i)
        gmag = np.abs(oracle.simulated_gradient(g_sim[i], "f32", ops[i], w.lam, SEED, 3, i))
        got = (host(p.data)[0], host(st["exp_avg"])[0], host(st["exp_avg_sq"])[0])
        for name, ok in zip(("theta", "exp_avg", "exp_avg_sq"), check_adam(got, old[i], f64, hp, gmag)):
            assert ok.all(), f"{w.names[i]} {name}: {np.count_nonzero(~ok)} mismatches"
    # the torch optimizer carries on from the state the fused step left
    opt.zero_grad()
    assert not w.begin(4)
    model.loss(batches[0]).backward()
    opt.step()
    assert all(int(float(opt.state[p]["step"])) == 5 for p in w.params)
    w.close()


def test_fused_clipped_step_matches_oracle():
    """end(fused=True, max_norm) clips the expert gradient to max_norm before the AdamW update, with
    the factor computed and applied on the GPU; the returned norm is the gradient's total norm."""
    model = make_decoder(TINY, 37, DEV)
    w = wrap(model)
    opt = torch.optim.AdamW(w.params, lr=1e-3, betas=(0.9, 0.95), weight_decay=1e-3)
    gen = torch.Generator(DEV).manual_seed(2)
    for p in w.params:                                   # a state as after a few steps
        opt.state[p] = dict(step=torch.tensor(3.0), exp_avg=torch.randn(p.shape, device=DEV, generator=gen) * 1e-3,
                            exp_avg_sq=torch.rand(p.shape, device=DEV, generator=gen) * 1e-6)
    assert w.begin(3)
    model.loss(token_batches(TINY, 2, 16, 1, 5, DEV)[0]).backward()
    old = [(host(m)[0], host(opt.state[p]["exp_avg"])[0], host(opt.state[p]["exp_avg_sq"])[0])
           for p, m in zip(w.params, w.master)]
    g_sim = [host(p.grad)[0] for p in w.params]    # the gradients at theta~ autograd produced
    ops = [op(w, i) for i in range(len(w.params))]
    sq = sum(oracle.grad_sqnorm(g_sim[i], "f32", ops[i], w.lam, SEED, 3, i) for i in range(len(g_sim)))
    max_norm = 0.25 * float(np.sqrt(sq))
    norm = w.end(opt, fused=True, max_norm=max_norm)
    torch.cuda.synchronize()
    assert check_sqnorm(float(norm.item()) ** 2, sq, sq * (1 + 1e-6))
    coef = float(w._clip[1].item())
    assert abs(coef - oracle.clip_coefficient(np.sqrt(sq), max_norm)) <= (0.5 * SQNORM_ULPS + 2) * U * coef
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=1e-3, grad_scale=coef, step=4)
    for i, p in enumerate(w.params):
        st = opt.state[p]
        _, f64 = oracle.adamw_fused(g_sim[i], "f32", *old[i], ops[i], w.lam, hp, SEED, 3, i)
        gmag = coef * np.abs(oracle.simulated_gradient(g_sim[i], "f32", ops[i], w.lam, SEED, 3, i))
        got = (host(p.data)[0], host(st["exp_avg"])[0], host(st["exp_avg_sq"])[0])
        for name, ok in zip(("theta", "exp_avg", "exp_avg_sq"), check_adam(got, old[i], f64, hp, gmag)):
            assert ok.all(), f"{w.names[i]} {name}: {np.count_nonzero(~ok)} mismatches"
    w.close()


@pytest.mark.parametrize("fused", [False, True])
def test_mixed_objective_adds_both_gradients(fused):
    """With the expert loss's backward before begin(), the simulated-loss gradient is added to it:
    grad = g_expert + lam alpha m g~ (Eq. smat-objective with both losses in one step)."""
    model = make_decoder(TINY, 43, DEV)
    batches = token_batches(TINY, 2, 16, 2, 3, DEV)
    lam = 0.25
    w = wrap(model, lam=lam, period=1)
    opt = torch.optim.AdamW(w.params, lr=1e-3, weight_decay=0.0)
    ((1 - lam) * model.loss(batches[0])).backward()            # expert loss at theta
    g_exp = [host(p.grad)[0] for p in w.params]
    masters = [host(m)[0] for m in w.master]
    assert w.begin(0)
    model.loss(batches[1]).backward()                           # simulated loss at theta~
    g_sim = [host(p.grad)[0] for p in w.params]
    ops = [op(w, i) for i in range(len(w.params))]
    w.end(opt, fused=fused)
    torch.cuda.synchronize()
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, grad_scale=1.0, step=1)
    for i, p in enumerate(w.params):
        if not fused:
            want = oracle.backward_accum(g_sim[i], "f32", g_exp[i], ops[i], lam, SEED, 0, i)
            incr = np.abs(oracle.simulated_gradient(g_sim[i], "f32", ops[i], lam, SEED, 0, i))
            ok = check_grad(host(p.grad)[0], want, g_exp[i], incr)
            assert ok.all(), f"{w.names[i]}: {np.count_nonzero(~ok)} gradient mismatches"
        else:
            old = (masters[i], np.zeros(p.numel(), np.float32), np.zeros(p.numel(), np.float32))
            _, f64 = oracle.adamw_fused(g_sim[i], "f32", *old, ops[i], lam, hp, SEED, 0, i, grad_acc=g_exp[i])
            gmag = np.abs(oracle.simulated_gradient(g_sim[i], "f32", ops[i], lam, SEED, 0, i)) + np.abs(g_exp[i])
            st = opt.state[p]
            got = (host(p.data)[0], host(st["exp_avg"])[0], host(st["exp_avg_sq"])[0])
            for name, ok in zip(("theta", "exp_avg", "exp_avg_sq"), check_adam(got, old, f64, hp, gmag)):
                assert ok.all(), f"{w.names[i]} {name}: {np.count_nonzero(~ok)} mismatches"
    # abort() puts the expert loss's gradients back
    ((1 - lam) * model.loss(batches[0])).backward()
    before = [p.grad.clone() for p in w.params]
    assert w.begin(1)
    w.abort()
    assert all(torch.equal(p.grad, b) for p, b in zip(w.params, before))
    w.close()


def test_fused_update_creates_missing_optimizer_state():
    model = make_decoder(TINY, 13, DEV)
    w = wrap(model, period=1)                       # every step simulated
    opt = torch.optim.AdamW(w.params, lr=1e-3, weight_decay=0.0)
    masters = [p.detach().clone() for p in w.params]
    assert w.begin(0)
    model.loss(token_batches(TINY, 2, 8, 1, 1, DEV)[0]).backward()
    g_sim = [host(p.grad)[0] for p in w.params]    # the gradients at theta~ autograd produced
    ops = [op(w, i) for i in range(len(w.params))]
    w.end(opt, fused=True)
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, grad_scale=1.0, step=1)
    for i, p in enumerate(w.params):
        st = opt.state[p]
        assert set(st) == {"step", "exp_avg", "exp_avg_sq"} and int(float(st["step"])) == 1
        old = (host(masters[i])[0], np.zeros(p.numel(), np.float32), np.zeros(p.numel(), np.float32))
        _, f64 = oracle.adamw_fused(g_sim[i], "f32", *old, ops[i], w.lam, hp, SEED, 0, i)
        got = (host(p.data)[0], host(st["exp_avg"])[0], host(st["exp_avg_sq"])[0])
        assert all(ok.all() for ok in check_adam(got, old, f64, hp))
    w.close()


def test_offload_reproduces_resident_across_cycles():
    """Two wrappers over the same parameters, one with theta0 resident and one prefetching it
    from pinned host memory: theta~ must agree bit for bit on every simulated step, with
    optimizer steps changing the expert weights in between."""
    model = make_decoder(TINY, 17, DEV)
    batches = token_batches(TINY, 2, 16, 12, 19, DEV)
    res = wrap(model, buffer_dtype=torch.bfloat16)
    off = wrap(model, buffer_dtype=torch.bfloat16, offload=True)
    opt = torch.optim.AdamW(res.params, lr=1e-2)
    for step in range(12):
        opt.zero_grad()
        if res.begin(step):
            a = [b.clone() for b in res.buffers]
            res.abort()
            assert off.begin(step)
            assert off.alpha == res.alpha
            for x, y in zip(a, off.buffers):
                assert torch.equal(x.view(torch.int16), y.view(torch.int16))
            check_simulated(off, [m.clone() for m in off.master], step)
            off.abort()
        else:
            assert not off.begin(step)
        model.loss(batches[step]).backward()
        opt.step()
    res.close()
    off.close()


def test_bf16_autocast_loop_runs():
    model = make_decoder(TINY, 23, DEV)
    batches = token_batches(TINY, 4, 32, 8, 29, DEV)
    w = SimulatedMergeTraining.from_module(model, seed=SEED, buffer_dtype=torch.bfloat16)
    opt = torch.optim.AdamW(w.params, lr=1e-3, weight_decay=0.01, fused=True)
    masters = [p.data for p in w.params]
    losses = []
    for step in range(8):
        opt.zero_grad()
        sim = w.begin(step)
        if sim:
            assert all(p.dtype == torch.bfloat16 for p in w.params)
            check_simulated(w, [m.clone() for m in masters], step)
        with torch.autocast("cuda", dtype=torch.bfloat16):
            loss = model.loss(batches[step])
        loss.backward()
        losses.append(float(loss.detach()))
        if sim:
            w.end(opt, fused=(step == 7))
            assert all(p.dtype == torch.float32 and p.data_ptr() == m.data_ptr() for p, m in zip(w.params, masters))
            if step == 7:
                continue
        opt.step()
    assert np.isfinite(losses).all()
    assert all(int(float(opt.state[p]["step"])) == 8 for p in w.params)
    w.close()


def test_wrapper_errors():
    model = make_decoder(TINY, 31, DEV)
    w = wrap(model)
    with pytest.raises(smat.SmatError):
        w.end()                                    # no open simulated step
    assert w.begin(3)
    with pytest.raises(smat.SmatError):
        w.begin(7)                                 # one already open
    with pytest.raises(smat.SmatError):
        w.end(torch.optim.SGD(w.params, lr=0.1), fused=True)
    extra = torch.nn.Parameter(torch.zeros(3, device=DEV))
    extra.grad = torch.ones(3, device=DEV)
    with pytest.raises(smat.SmatError):            # a parameter the fused update would skip
        w.end(torch.optim.AdamW(w.params + [extra], lr=1e-3), fused=True)
    assert w.active                                # a rejected end() leaves the step open
    w.abort()
    assert not w.active and all(p.data_ptr() == m.data_ptr() for p, m in zip(w.params, w.master))
    w.abort()                                      # idempotent
    with pytest.raises(smat.SmatError):
        SimulatedMergeTraining([torch.nn.Parameter(torch.zeros(4, device=DEV, dtype=torch.bfloat16))],
                               [torch.zeros(4, device=DEV)], [1.0], 0.2, 1e-3)
    w.close()


def test_micro_batches_accumulate_in_a_simulated_step():
    """Gradient accumulation inside a simulated step: several forward/backward passes on theta~
    accumulate into the gradient at theta~ (autograd adds into p.grad), and end() turns the sum into
    the expert gradient lam alpha m (.) (sum of g~) for the optimizer."""
    torch.manual_seed(0)
    model = make_decoder(TINY, 5, DEV)
    batches = token_batches(TINY, 2, 24, 3, 11, DEV)
    w = wrap(model)
    assert w.begin(3)
    for tokens in batches:                              # three micro-batches
        (model.loss(tokens) / len(batches)).backward()
    g_sum = [host(p.grad)[0] for p in w.params]         # what autograd accumulated at theta~
    # the same sum from a copy of the model holding theta~
    ref = make_decoder(TINY, 5, DEV)
    with torch.no_grad():
        for q, p in zip(ref.parameters(), w.params):
            q.copy_(p.data)
    for tokens in batches:
        (ref.loss(tokens) / len(batches)).backward()
    for p, q in zip(w.params, ref.parameters()):
        torch.testing.assert_close(p.grad, q.grad, rtol=1e-5, atol=1e-7)
    w.end()
    for i, p in enumerate(w.params):
        zeros = np.zeros(p.numel(), np.float32)
        want = oracle.backward_accum(g_sum[i], "f32", zeros, op(w, i), w.lam, SEED, 3, i)
        incr = np.abs(oracle.simulated_gradient(g_sum[i], "f32", op(w, i), w.lam, SEED, 3, i))
        assert check_grad(host(p.grad)[0], want, zeros, incr).all(), w.names[i]
    w.close()
