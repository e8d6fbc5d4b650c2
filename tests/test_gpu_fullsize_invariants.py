"""Every element of the full-size lists, launched as the benchmark launches them (one plan, one
simulate and one backward launch over the whole list), checked by properties that hold at any size.

With s = 1, no 1/keep rescale and no noise, Eq. smat-state leaves a kept coordinate at theta (the
lerp with t = 1 is exact in fp32) and a dropped one at theta0, so every simulated weight is either
bf16(theta) or theta0 (Sec. 4.1, Eq. smat-mask).  Eq. smat-gradient with t = 1 adds lambda g~ on
the kept coordinates and leaves the dropped ones alone.  The mask is the same draw in both kernels
(Sec. 4.2: regenerated, never stored), so for every element

* theta~ is bf16(theta) or theta0 (torch's own round-to-nearest-even conversion gives bf16(theta));
* where bf16(theta) != theta0 the element is classified: kept => grad_theta == fl32(grad_theta +
  lambda g~) bit for bit (one rounding, as a fused multiply-add rounds), dropped => grad_theta keeps
  its bits;
* where bf16(theta) == theta0 the element cannot be classified from theta~, and grad_theta holds one
  of the two values;
* the dropped fraction among classified elements of a masked tensor is Binomial(n, 1 - keep)
  (classification depends on the data only, the mask on the counter-based draw), checked at 6
  standard deviations per tensor and over the list.

The sampled windows of the same lists are compared with the oracle in test_gpu_fullsize.py; this
test covers the elements between them."""
import math

import numpy as np
import pytest
import torch

import paper_2609_33437_amd as smat
import workloads

pytestmark = pytest.mark.gpu
DEV = "cuda"
NAN_BF16 = 0x7FC0


def _bits32(x):
    return x.view(torch.int32)


@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5"])
def test_fullsize_every_element_invariants(name):
    cfg = workloads.config(name)
    print(f"[{name}] generating {cfg.count} tensors, {cfg.numel} params", flush=True)
    inp = workloads.make_inputs(cfg, device=DEV)
    # sentinel: an element the simulate never wrote stays NaN, which is neither bf16(theta) nor theta0
    outs = [torch.full((t.numel(),), NAN_BF16, dtype=torch.int16, device=DEV).view(torch.bfloat16)
            for t in inp.theta]
    step = 5
    params = [dict(p, s=1.0, rescale=0, sigma=0.0) for p in workloads.step_params(cfg, inp.settings, step)]
    lam = float(np.float32(cfg.lam))
    g_old = [g.clone() for g in inp.grad_theta]
    with smat.Plan(inp.theta, outs, inp.theta0, inp.grad_sim, inp.grad_theta) as plan:
        plan.set_params(params)
        plan.simulate(cfg.smat_seed, step)
        plan.switch_storage(smat.SMAT_SIMULATED)
        plan.backward_accum(cfg.smat_seed, step, lam)
        plan.switch_storage(smat.SMAT_EXPERT)
        torch.cuda.synchronize()
    print(f"[{name}] kernels done, checking every element", flush=True)
    tot_n = tot_drop = 0
    tot_mean = tot_var = 0.0
    n_amb = 0
    for i in range(cfg.count):
        what = f"{name} tensor {i} ({cfg.specs[i].name})"
        keep = params[i]["keep"]
        th = inp.theta[i].view(-1)
        t0 = inp.theta0[i].view(-1)
        out = outs[i]
        r = th.to(torch.bfloat16)
        is_r, is_t0 = out == r, out == t0
        assert bool((is_r | is_t0).all()), f"{what}: theta~ neither bf16(theta) nor theta0"
        amb = r == t0
        dropped = is_t0 & ~amb
        kept = is_r & ~amb
        gn, go = inp.grad_theta[i].view(-1), g_old[i].view(-1)
        want = (go.double() + lam * inp.grad_sim[i].view(-1).double()).float()
        same_old, same_want = _bits32(gn) == _bits32(go), _bits32(gn) == _bits32(want)
        assert bool(same_old[dropped].all()), f"{what}: a dropped coordinate's gradient changed"
        assert bool(same_want[kept].all()), f"{what}: a kept coordinate's gradient is not g + lambda g~"
        assert bool((same_old | same_want)[amb].all()), f"{what}: gradient neither kept nor dropped"
        n = int((~amb).sum())
        d = int(dropped.sum())
        n_amb += int(amb.sum())
        if keep >= 1.0:
            assert d == 0, f"{what}: keep = 1 dropped {d} coordinates"
            continue
        p = 1.0 - math.floor(keep * 2.0 ** 32) / 2.0 ** 32
        sd = math.sqrt(n * p * (1.0 - p))
        assert abs(d - n * p) <= 6.0 * sd + 1.0, f"{what}: {d} of {n} dropped, expected {n * p:.0f} +- {sd:.0f}"
        tot_n, tot_drop = tot_n + n, tot_drop + d
        tot_mean, tot_var = tot_mean + n * p, tot_var + n * p * (1.0 - p)
        del r, is_r, is_t0, amb, dropped, kept, want, same_old, same_want
    print(f"[{name}] {cfg.numel} elements: {n_amb} unclassifiable (bf16(theta) == theta0), "
          f"{tot_drop} of {tot_n} classified masked elements dropped (expected {tot_mean:.0f} "
          f"+- {math.sqrt(tot_var):.0f})", flush=True)
    assert abs(tot_drop - tot_mean) <= 6.0 * math.sqrt(tot_var) + 1.0
    del inp, outs, g_old
    torch.cuda.empty_cache()
