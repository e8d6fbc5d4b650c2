"""smat_simulate_multi_static, the list simulate that allocates nothing (its tables live in a static
device array of the library), against the plan-based smat_simulate_multi: the same output bits on
ragged lists, on two calls in a row whose second list is smaller than the first, and its limits."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2609_33437_amd as smat
from paper_2609_33437_amd import _lib

DEV = "cuda"


def _descs(thetas, theta0s, outs, ids, offs):
    d = (_lib.smat_tensor_desc * max(len(thetas), 1))()
    for i, (th, t0, o) in enumerate(zip(thetas, theta0s, outs)):
        d[i].theta = ctypes.c_void_p(th.data_ptr()) if th.numel() else None
        d[i].theta0 = ctypes.c_void_p(t0.data_ptr()) if t0.numel() else None
        d[i].out = ctypes.c_void_p(o.data_ptr()) if o.numel() else None
        d[i].n = th.numel()
        d[i].tensor_id = ids[i]
        d[i].elem_offset = offs[i]
    return d


def _ragged(gen, sizes, dt, misalign=()):
    """theta (fp32), theta0 and two output buffers per size; tensors listed in `misalign` start one
    element into their allocation, so their quads do not line up with 16-byte vectors."""
    th, t0, out_a, out_b = [], [], [], []
    for i, n in enumerate(sizes):
        k = 1 if i in misalign else 0
        a = torch.randn(n + k, device=DEV, generator=gen)[k:] * 0.02
        b = (a + torch.randn(n, device=DEV, generator=gen) * 1e-3).to(dt)
        b = torch.cat([b.new_zeros(k), b])[k:] if k else b
        th.append(a)
        t0.append(b)
        out_a.append(torch.full((n + k,), float("nan"), device=DEV, dtype=dt)[k:])
        out_b.append(torch.full((n + k,), float("nan"), device=DEV, dtype=dt)[k:])
    return th, t0, out_a, out_b


def _params(rng, count):
    keep = rng.choice([0.0, 0.25, 0.5, 0.9, 1.0], size=count)
    sigma = rng.choice([0.0, 1e-3], size=count)
    return smat.op_params_array(count, rng.uniform(0.2, 1.0, size=count).astype(np.float32), keep.astype(np.float32),
                                sigma.astype(np.float32), rescale=rng.integers(0, 2, size=count).astype(np.int32),
                                noise_kind=rng.integers(0, 3, size=count).astype(np.int32))


def _static(th, t0, out, ids, offs, params, seed, step):
    lib = smat.lib()
    d = _descs(th, t0, out, ids, offs)
    dt = _lib.dtype_code(out[0])
    st = lib.smat_simulate_multi_static(d, len(th), _lib.dtype_code(t0[0]), dt,
                                        params.ctypes.data_as(ctypes.POINTER(_lib.smat_op_params)), seed, step,
                                        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, lib.smat_last_error().decode()


def _planned(th, t0, out, ids, offs, params, seed, step):
    with smat.Plan(th, out, t0, tensor_ids=ids, elem_offsets=offs) as plan:
        plan.set_params(params)
        plan.simulate(seed, step)
        torch.cuda.synchronize()


def _same_bits(a, b):
    for i, (x, y) in enumerate(zip(a, b)):
        assert torch.equal(x.view(torch.int16), y.view(torch.int16)), f"tensor {i} differs"


@pytest.mark.gpu
def test_static_list_matches_the_plan_on_two_calls_the_second_smaller():
    gen = torch.Generator(DEV).manual_seed(11)
    rng = np.random.default_rng(11)
    # first call: 12 tensors over several chunks, ragged tails, odd offsets, misaligned bases
    sizes = [1, 3, 257, 16384, 3 * 16384 + 7, 100_000, 1792, 5, 65536, 40_001, 16383, 2 * 16384]
    offs = [0, 5, 0, 4, 0, 3, 0, 0, (1 << 33) + 8, 2, 0, 0]
    th, t0, out_s, out_p = _ragged(gen, sizes, torch.bfloat16, misalign=(2, 7))
    ids = list(range(100, 100 + len(sizes)))
    params = _params(rng, len(sizes))
    _static(th, t0, out_s, ids, offs, params, seed=0x5EED, step=7)
    _planned(th, t0, out_p, ids, offs, params, seed=0x5EED, step=7)
    torch.cuda.synchronize()
    _same_bits(out_s, out_p)
    # second call, on the same stream right after the first: a smaller list in fp32
    sizes2 = [4099, 20_000, 9]
    th2, t02, out_s2, out_p2 = _ragged(gen, sizes2, torch.float32)
    params2 = _params(rng, len(sizes2))
    _static(th, t0, out_s, ids, offs, params, seed=0x5EED, step=8)    # the first list again, new step
    _static(th2, t02, out_s2, [0, 1, 2], [0, 0, 0], params2, seed=3, step=1 << 29)
    _planned(th2, t02, out_p2, [0, 1, 2], [0, 0, 0], params2, seed=3, step=1 << 29)
    _planned(th, t0, out_p, ids, offs, params, seed=0x5EED, step=8)
    torch.cuda.synchronize()
    _same_bits(out_s2, out_p2)
    _same_bits(out_s, out_p)
    # every element was written (the buffers started as NaN and the inputs are finite)
    for o in out_s + out_s2:
        assert not bool(torch.isnan(o.float()).any())


def test_static_list_rejects_lists_beyond_its_tables():
    """Host-side checks: they fail before any HIP call (the descriptors below point nowhere)."""
    lib = smat.lib()
    p = smat.op_params_array(1, 1.0, 1.0, 0.0)
    pp = p.ctypes.data_as(ctypes.POINTER(_lib.smat_op_params))
    many = (_lib.smat_tensor_desc * 8193)()
    many_p = smat.op_params_array(8193, 1.0, 1.0, 0.0)
    st = lib.smat_simulate_multi_static(many, 8193, _lib.SMAT_BF16, _lib.SMAT_BF16,
                                        many_p.ctypes.data_as(ctypes.POINTER(_lib.smat_op_params)), 0, 0, None)
    assert st == _lib.SMAT_ERR_INVALID and b"at most 8192" in lib.smat_last_error()
    # one tensor of 2^34 elements needs 2^20 chunks, more than the 8 MiB array holds
    big = (_lib.smat_tensor_desc * 1)()
    big[0].theta, big[0].theta0, big[0].out = 1 << 44, 2 << 44, 3 << 44
    big[0].n = 1 << 34
    st = lib.smat_simulate_multi_static(big, 1, _lib.SMAT_BF16, _lib.SMAT_BF16, pp, 0, 0, None)
    assert st == _lib.SMAT_ERR_INVALID and b"use a plan" in lib.smat_last_error()
    # the plan's argument rules apply: aliasing and params are checked
    big[0].n = 1000
    big[0].out = big[0].theta
    st = lib.smat_simulate_multi_static(big, 1, _lib.SMAT_BF16, _lib.SMAT_BF16, pp, 0, 0, None)
    assert st == _lib.SMAT_ERR_INVALID
    big[0].out = 3 << 44
    bad = smat.op_params_array(1, 1.0, 1.5, 0.0)
    st = lib.smat_simulate_multi_static(big, 1, _lib.SMAT_BF16, _lib.SMAT_BF16,
                                        bad.ctypes.data_as(ctypes.POINTER(_lib.smat_op_params)), 0, 0, None)
    assert st == _lib.SMAT_ERR_INVALID
    st = lib.smat_simulate_multi_static(big, 1, _lib.SMAT_BF16, _lib.SMAT_BF16, pp, 0, 1 << 30, None)
    assert st == _lib.SMAT_ERR_INVALID
