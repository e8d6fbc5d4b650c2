"""The Python binding's size and dtype checks (CPU, no GPU call is reached): the C ABI receives only
pointers and element counts, so an array shorter or narrower than the launch assumes would be
overrun by a kernel.  Every case here must be refused before the library is called."""
import pytest
import torch

import paper_2609_33437_amd as smat
from paper_2609_33437_amd._lib import SMAT_BF16, SMAT_ERR_DTYPE, SMAT_ERR_INVALID, SMAT_F32, _expect

F32, BF16 = torch.float32, torch.bfloat16


def status_of(fn):
    with pytest.raises(smat.SmatError) as e:
        fn()
    return e.value.status


def test_expect_checks_count_and_dtype():
    _expect(torch.zeros(5), 5, SMAT_F32, "x")
    _expect(None, 5, SMAT_F32, "x")
    assert status_of(lambda: _expect(torch.zeros(4), 5, SMAT_F32, "x")) == SMAT_ERR_INVALID
    assert status_of(lambda: _expect(torch.zeros(5, dtype=BF16), 5, SMAT_F32, "x")) == SMAT_ERR_DTYPE
    assert status_of(lambda: _expect(torch.zeros(5), 5, SMAT_BF16, "x")) == SMAT_ERR_DTYPE
    assert status_of(lambda: _expect(torch.zeros(5, dtype=torch.float16), 5, SMAT_F32, "x")) == SMAT_ERR_DTYPE


def test_single_tensor_entry_points():
    n = 8
    th, t0, out = torch.zeros(n), torch.zeros(n, dtype=BF16), torch.zeros(n, dtype=BF16)
    p = dict(s=1.0, keep=1.0, sigma=0.0)
    # theta must be fp32: a bf16 theta would be read as 4 n bytes
    assert status_of(lambda: smat.smat_simulate(th.to(BF16), t0, out, p, 0, 0)) == SMAT_ERR_DTYPE
    assert status_of(lambda: smat.smat_simulate(th, t0[:7], out, p, 0, 0)) == SMAT_ERR_INVALID
    # grad_theta must be fp32
    assert status_of(lambda: smat.smat_backward_accum(t0, out, p, 1.0, 0, 0)) == SMAT_ERR_DTYPE
    # the optimizer arrays must be fp32 and of theta's size
    m = torch.zeros(n)
    assert status_of(lambda: smat.smat_adamw_fused(t0, th, m[:7], m, p, 1.0, {}, 0, 0)) == SMAT_ERR_INVALID
    assert status_of(lambda: smat.smat_adamw_fused(t0, th, m.to(BF16), m, p, 1.0, {}, 0, 0)) == SMAT_ERR_DTYPE
    # debug draws: 4-byte words, 1-byte flags, fp32 z
    assert status_of(lambda: smat.smat_debug_draws(n, p, 0, 0, mask_words=torch.zeros(n, dtype=torch.uint8))) \
        == SMAT_ERR_INVALID
    assert status_of(lambda: smat.smat_debug_draws(n, p, 0, 0, kept=torch.zeros(n, dtype=torch.int32))) \
        == SMAT_ERR_INVALID
    assert status_of(lambda: smat.smat_debug_draws(n, p, 0, 0, z=torch.zeros(n, dtype=torch.int32))) == SMAT_ERR_DTYPE


def test_plan_lists():
    th = [torch.zeros(8), torch.zeros(5)]
    t0 = [torch.zeros(8, dtype=BF16), torch.zeros(5, dtype=BF16)]
    out = [torch.zeros(8, dtype=BF16), torch.zeros(5, dtype=BF16)]
    gs = [torch.zeros(8, dtype=BF16), torch.zeros(5, dtype=BF16)]
    gt = [torch.zeros(8), torch.zeros(5)]
    # an fp32 buffer behind a bf16 first buffer, and the other way round
    assert status_of(lambda: smat.Plan(th, [out[0], torch.zeros(5)], t0, gs, gt)) == SMAT_ERR_DTYPE
    assert status_of(lambda: smat.Plan(th, [torch.zeros(8), out[1]], t0, gs, gt)) == SMAT_ERR_DTYPE
    # sizes that differ from theta's
    assert status_of(lambda: smat.Plan(th, out, [t0[0], t0[1][:4]], gs, gt)) == SMAT_ERR_INVALID
    assert status_of(lambda: smat.Plan(th, out, t0, [gs[0], gs[1][:4]], gt)) == SMAT_ERR_INVALID
    assert status_of(lambda: smat.Plan(th, out, t0, gs, [gt[0], gt[1].to(BF16)])) == SMAT_ERR_DTYPE
    assert status_of(lambda: smat.Plan([th[0], th[1].to(BF16)], out, t0, gs, gt)) == SMAT_ERR_DTYPE
    # lists of different lengths
    assert status_of(lambda: smat.Plan(th, out[:1], t0, gs, gt)) == SMAT_ERR_INVALID
    assert status_of(lambda: smat.Plan(th, out, t0, gs, gt, tensor_ids=[0])) == SMAT_ERR_INVALID
    # explicit dtypes are checked against the arrays too
    assert status_of(lambda: smat.Plan(th, out, t0, gs, gt, dtypes=(SMAT_F32, SMAT_BF16, SMAT_BF16))) \
        == SMAT_ERR_DTYPE


def test_merge_lists():
    t0 = [torch.zeros(8, dtype=BF16), torch.zeros(5, dtype=BF16)]
    ex = [[torch.zeros(8, dtype=BF16), torch.zeros(5, dtype=BF16)]]
    assert status_of(lambda: smat.MergePlan(t0, [torch.zeros(8, dtype=BF16), torch.zeros(5)], ex)) == SMAT_ERR_DTYPE
    assert status_of(lambda: smat.MergePlan([t0[0], torch.zeros(5)], [x.clone() for x in t0], ex)) == SMAT_ERR_DTYPE
    assert status_of(lambda: smat.MergePlan(t0, [x.clone() for x in t0], [[ex[0][0], ex[0][1][:4]]])) \
        == SMAT_ERR_INVALID
    assert status_of(lambda: smat.MergePlan(t0, [x.clone() for x in t0], [[ex[0][0], ex[0][1].float()]])) \
        == SMAT_ERR_DTYPE


def test_op_params_array_matches_the_c_records():
    import ctypes
    import numpy as np
    from paper_2609_33437_amd import _lib
    keeps, kinds = [0.1, 1.0, 0.0, 0.37], [0, 1, 2, 0]
    a = smat.op_params_array(4, 0.5, keeps, [1e-3, 0.0, 2e-3, 5e-4], [1, 0, 1, 1], kinds)
    recs = (_lib.smat_op_params * 4)(*[_lib.op_params(dict(s=0.5, keep=k, sigma=sg, rescale=r, noise_kind=nk))
                                       for k, sg, r, nk in zip(keeps, [1e-3, 0.0, 2e-3, 5e-4], [1, 0, 1, 1], kinds)])
    assert a.tobytes() == ctypes.string_at(recs, ctypes.sizeof(recs))
    assert smat.OP_PARAMS_DTYPE.itemsize == ctypes.sizeof(_lib.smat_op_params)
    assert np.all(a["keep"] == np.float32(keeps))
