"""The simulate's choice between its vector path and its element-by-element path, at the edges of
the static whole-tensor flag: that flag needs quad-aligned pointers, n a multiple of 4 and an
element offset that is a multiple of the 256-element tile.  Tensors just inside and just outside
each condition (n = 1024 / 1023 / 1026, offsets 0 / 4 / 252 / 256 / 260 / 2^34 - 8, a misaligned
base), in one list launch, every element compared with the oracle (Sec. 4.1, Eq. smat-state, with
mask and Gaussian noise; Sec. 4.2, Eq. smat-gradient).  Both paths compute the same arithmetic, so
each must meet the same bar."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_33437_amd as smat
from helpers import host
from tolerances import check_grad, check_theta_tilde

pytestmark = pytest.mark.gpu
DEV = "cuda"
SEED, STEP, LAM = 0x5EED, 11, 0.75
P = dict(s=0.8, keep=0.4, sigma=3e-3, rescale=1, noise_kind=0)

# (n, element offset, extra leading elements that misalign the base pointers)
CASES = [(1024, 0, 0), (1023, 0, 0), (1026, 0, 0), (1024, 4, 0), (1024, 252, 0), (1024, 256, 0),
         (1024, 260, 0), (4096, 2 ** 34 - 8, 0), (4096, 2 ** 34 - 256, 0), (1024, 0, 1), (257, 0, 0),
         (3, 0, 0), (300000, 512, 0), (299999, 768, 0)]


def test_vector_path_edges_in_one_list():
    gen = torch.Generator().manual_seed(7)
    th, t0, gs, gt, out, keep_alive = [], [], [], [], [], []
    for n, _, shift in CASES:
        base_t = (torch.randn(n + shift, generator=gen) * 0.02)
        base_0 = (base_t + torch.randn(n + shift, generator=gen) * 1e-3).to(torch.bfloat16)
        g = (torch.randn(n + shift, generator=gen) * 1e-2).to(torch.bfloat16)
        a = (torch.randn(n + shift, generator=gen) * 1e-3)
        dev = [x.to(DEV) for x in (base_t, base_0, g, a)]
        keep_alive.append(dev)
        th.append(dev[0][shift:])
        t0.append(dev[1][shift:])
        gs.append(dev[2][shift:])
        gt.append(dev[3][shift:])
        out.append(torch.full((n,), 0x7FC0, dtype=torch.int16, device=DEV).view(torch.bfloat16))
    inputs = [(host(th[i])[0], host(t0[i])[0], host(gs[i])[0], host(gt[i])[0]) for i in range(len(CASES))]
    offs = [off for _, off, _ in CASES]
    with smat.Plan(th, out, t0, gs, gt, elem_offsets=offs) as plan:
        plan.set_params([P] * len(CASES))
        plan.simulate(SEED, STEP)
        plan.switch_storage(smat.SMAT_SIMULATED)
        plan.backward_accum(SEED, STEP, LAM)
        plan.switch_storage(smat.SMAT_EXPERT)
        torch.cuda.synchronize()
    for i, (n, off, shift) in enumerate(CASES):
        what = f"tensor {i}: n={n} offset={off} shift={shift}"
        thn, t0n, gsn, g_old = inputs[i]
        y, kept, eps = oracle.simulate_f64(thn, t0n, "bf16", P, SEED, STEP, i, off)
        coef = np.where(kept, oracle.coefficient(P["s"], P["keep"], P["rescale"]), 0.0)
        ok, _ = check_theta_tilde(host(out[i])[0], "bf16", y, thn, oracle.as_f64(t0n, "bf16"), coef, eps, P["sigma"])
        assert ok.all(), f"{what}: {np.count_nonzero(~ok)} theta~ mismatches"
        want = oracle.backward_accum(gsn, "bf16", g_old, P, LAM, SEED, STEP, i, off)
        got = host(gt[i])[0]
        assert check_grad(got, want, g_old, np.abs(LAM * coef * oracle.as_f64(gsn, "bf16"))).all(), f"{what}: grad"
        np.testing.assert_array_equal(got.view(np.uint32)[~kept], g_old.view(np.uint32)[~kept], err_msg=what)
