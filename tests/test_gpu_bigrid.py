"""GPU tests of jobs whose one-launch grid would hold more than 2^32 work-items, which a dispatch
cannot express (the count would wrap without an error): the launchers split them into several
launches.  A copy of 68.7 GB, a one-tensor backward of 17.2e9 elements, 4.3e9 raw Philox words and
a list of 2.2 million tensors (2.2 million chunks) are checked against the oracle at the piece
boundaries and at the end, and for having written every element."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2609_33437_amd as smat
from paper_2609_33437_amd import _lib
from helpers import host
from tolerances import check_grad, check_theta_tilde

pytestmark = pytest.mark.gpu
DEV = "cuda"
MAX_BLOCKS = 0xFFFFFFFF // 64          # one-wave blocks per launch
GIB = 1 << 30


def free_gib():
    torch.cuda.empty_cache()
    return torch.cuda.mem_get_info()[0] / GIB


def test_stream_copy_past_the_grid_limit():
    n16 = MAX_BLOCKS * 64 + 12345                       # 16-byte vectors: two launches
    if free_gib() < 2 * n16 * 16 / GIB + 8:
        pytest.skip("needs about 140 GB of free device memory")
    n = n16 * 4
    src = torch.empty(n, dtype=torch.float32, device=DEV)
    piece = 1 << 30
    for off in range(0, n, piece):                      # distinct values in every piece of the check
        src[off:off + piece] = torch.arange(off % 1000003, off % 1000003 + min(piece, n - off), device=DEV,
                                            dtype=torch.float32)
    dst = torch.zeros_like(src)
    smat.smat_stream_copy(src, dst)
    torch.cuda.synchronize()
    for off in range(0, n, piece):
        assert torch.equal(src[off:off + piece], dst[off:off + piece]), off
    del src, dst
    torch.cuda.empty_cache()


def test_backward_one_past_the_grid_limit():
    boundary = MAX_BLOCKS * 256                         # first element of the second launch
    n = boundary + 4099                                 # and a ragged tail
    if free_gib() < n * 6 / GIB + 8:
        pytest.skip("needs about 110 GB of free device memory")
    gen = torch.Generator(DEV).manual_seed(5)
    gs = torch.randn(n, device=DEV, dtype=torch.bfloat16, generator=gen)
    gt = torch.full((n,), 0.25, device=DEV, dtype=torch.float32)
    p = dict(s=0.6, keep=0.5, sigma=0.0, rescale=1)
    lam, seed, step, tid = 0.5, 77, 3, 9
    smat.smat_backward_accum(gs, gt, p, lam, seed, step, tid)
    torch.cuda.synchronize()
    for lo, hi in ((0, 4096), (boundary - 4096, boundary + 4096), (n - 4099, n)):
        gsn, gs_dt = host(gs[lo:hi])
        g_old = np.full(hi - lo, 0.25, dtype=np.float32)
        want = oracle.backward_accum(gsn, gs_dt, g_old, p, lam, seed, step, tid, lo)
        got = host(gt[lo:hi])[0]
        coef = oracle.coefficient(p["s"], p["keep"], p["rescale"])
        assert check_grad(got, want, g_old, np.abs(lam * coef * oracle.as_f64(gsn, gs_dt))).all(), lo
        assert (got != 0.25).any(), lo                  # the range was reached
    del gs, gt
    torch.cuda.empty_cache()


def test_debug_draws_past_the_grid_limit():
    boundary = (0xFFFFFFFF // 256) * 256               # 256-thread blocks: first element of the second launch
    n = boundary + 1029
    if free_gib() < n * 4 / GIB + 8:
        pytest.skip("needs about 25 GB of free device memory")
    words = torch.zeros(n, dtype=torch.int32, device=DEV)
    seed, step, tid, off = 12345, 6, 3, 1 << 33
    smat.smat_debug_draws(n, dict(s=1.0, keep=1.0, sigma=0.0), seed, step, tid, off, mask_words=words)
    torch.cuda.synchronize()
    for lo, hi in ((0, 1024), (boundary - 2048, boundary + 1029), (n - 1029, n)):
        want = oracle.element_words(seed, step, tid, off + lo, hi - lo, 0)
        got = words[lo:hi].cpu().numpy().view(np.uint32)
        np.testing.assert_array_equal(got, want, err_msg=str(lo))
    del words
    torch.cuda.empty_cache()


def _list_plan(count, bufs):
    """A plan over `count` tensors of 4 elements each, views into flat buffers, built through the
    C ABI from one descriptor array (no per-tensor Python objects)."""
    th, t0, out, gs, gt = bufs
    desc = np.zeros(count, dtype=np.dtype([("theta", "<u8"), ("theta0", "<u8"), ("out", "<u8"), ("grad_sim", "<u8"),
                                           ("grad_theta", "<u8"), ("theta0_host", "<u8"), ("n", "<i8"),
                                           ("tensor_id", "<u4"), ("reserved", "<u4"), ("elem_offset", "<u8")]))
    assert desc.itemsize == ctypes.sizeof(_lib.smat_tensor_desc)
    i = np.arange(count, dtype=np.uint64)
    desc["theta"] = th.data_ptr() + i * 16
    desc["theta0"] = t0.data_ptr() + i * 8
    desc["out"] = out.data_ptr() + i * 8
    desc["grad_sim"] = gs.data_ptr() + i * 8
    desc["grad_theta"] = gt.data_ptr() + i * 16
    desc["n"] = 4
    desc["tensor_id"] = i.astype(np.uint32)
    lib = smat.lib()
    plan = ctypes.c_void_p()
    st = lib.smat_plan_create(desc.ctypes.data_as(ctypes.POINTER(_lib.smat_tensor_desc)), count, _lib.SMAT_BF16,
                              _lib.SMAT_BF16, _lib.SMAT_BF16, 0, ctypes.byref(plan))
    assert st == 0, lib.smat_last_error()
    nb = ctypes.c_size_t()
    assert lib.smat_plan_workspace_bytes(plan, ctypes.byref(nb)) == 0
    ws = torch.empty(nb.value, dtype=torch.uint8, device=DEV)
    assert lib.smat_plan_bind_workspace(plan, ctypes.c_void_p(ws.data_ptr()), nb.value, None) == 0
    return plan, ws


def test_list_of_two_million_tensors():
    count = 2_200_000                                   # 2.2M chunks: 3 simulate and 3 backward launches
    gen = torch.Generator(DEV).manual_seed(6)
    n = 4 * count
    th = torch.randn(n, device=DEV, generator=gen) * 0.02
    t0 = (th + torch.randn(n, device=DEV, generator=gen) * 1e-3).to(torch.bfloat16)
    out = torch.full((n,), float("nan"), device=DEV, dtype=torch.bfloat16)
    gs = (torch.randn(n, device=DEV, generator=gen) * 1e-2).to(torch.bfloat16)
    gt = torch.full((n,), float("nan"), device=DEV, dtype=torch.float32)
    lib = smat.lib()
    plan, ws = _list_plan(count, (th, t0, out, gs, gt))
    try:
        params = smat.op_params_array(count, s=0.7, keep=0.4, sigma=1e-4)
        assert lib.smat_plan_set_params(plan, params.ctypes.data_as(ctypes.POINTER(_lib.smat_op_params)), None) == 0
        seed, step, lam = 31, 8, 0.5
        assert lib.smat_simulate_multi(plan, seed, step, None) == 0
        assert lib.smat_backward_multi(plan, seed, step, lam, 0, None) == 0      # overwrite: writes every element
        sumsq = torch.zeros(1, dtype=torch.float64, device=DEV)
        assert lib.smat_grad_norm_multi(plan, seed, step, lam, 0, 1.0, ctypes.c_void_p(sumsq.data_ptr()), None,
                                        None) == 0
        torch.cuda.synchronize()
    finally:
        assert lib.smat_plan_destroy(plan) == 0
    assert bool(torch.isfinite(out).all()) and bool(torch.isfinite(gt).all())
    # the norm covers the same gradient that the overwrite wrote
    ref = float((gt.double() ** 2).sum())
    assert abs(sumsq.item() - ref) <= 1e-5 * ref
    p = dict(s=float(np.float32(0.7)), keep=float(np.float32(0.4)), sigma=float(np.float32(1e-4)), rescale=1)
    sim_cut, bwd_cut = MAX_BLOCKS // 64, MAX_BLOCKS // 64      # chunks per simulate / backward launch
    picks = sorted(set(list(range(0, 40)) + list(range(sim_cut - 40, sim_cut + 40)) +
                       list(range(bwd_cut - 40, bwd_cut + 40)) + list(range(2 * bwd_cut - 40, 2 * bwd_cut + 40)) +
                       list(range(count - 40, count))))
    thn, t0n, outn, gsn, gtn = (host(x)[0] for x in (th, t0, out, gs, gt))
    for i in picks:
        e = slice(4 * i, 4 * i + 4)
        y, kept, eps = oracle.simulate_f64(thn[e], t0n[e], "bf16", p, seed, step, i)
        coef = np.where(kept, oracle.coefficient(p["s"], p["keep"], p["rescale"]), 0.0)
        ok, _ = check_theta_tilde(outn[e], "bf16", y, thn[e], oracle.as_f64(t0n[e], "bf16"), coef, eps, p["sigma"])
        assert ok.all(), i
        want = oracle.backward_accum(gsn[e], "bf16", np.zeros(4, np.float32), p, lam, seed, step, i)
        incr = np.abs(lam * coef * oracle.as_f64(gsn[e], "bf16"))
        assert check_grad(gtn[e], want, np.zeros(4, np.float32), incr).all(), i
