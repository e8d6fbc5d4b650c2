"""The storage switch against the oracle's state machine (Sec. 4.3, "Parameter storage switching";
App. "Implementation details"): one seeded random sequence of simulates, switches to either
storage, misuse (a switch to the simulated storage without a fresh simulate or twice in a row, a
simulate while the simulated storage is active, an unknown target, a step out of range) drives
oracle.StorageSwitch and a plan side by side, in resident and in offload mode.  After every call
the status codes, the storage state, the active pointers (host list and device table) and the bytes
of the active storage and of the buffers must agree.  The parameters (s = 1 without rescale, sigma =
0, keep in {0, 1/2, 1}) make every simulated value exact (theta rounded to bf16 where kept, theta0
where dropped), so the buffers are compared bit for bit while the mask draws still change with the
step."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2609_33437_amd as smat
from paper_2609_33437_amd import _lib

pytestmark = pytest.mark.gpu
DEV = "cuda"
SIZES = [1, 7, 256, 1000, 4099, 16384 + 5]
SEED = 0x5171C4
OPS = 300


def _inputs(gen):
    th, t0 = [], []
    for n in SIZES:
        b = (torch.randn(n, generator=gen) * 0.02).to(torch.bfloat16)
        th.append((b.float() + torch.randn(n, generator=gen) * 1e-3).contiguous())
        t0.append(b.contiguous())
    return th, t0


def _bits(t):
    t = t.detach().cpu()
    return t.view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.numpy().view(np.uint32)


def _np_bits(a):
    a = np.asarray(a)
    return a.view(np.uint16) if a.dtype == np.uint16 else a.astype(np.float32).view(np.uint32)


@pytest.mark.parametrize("offload", [False, True])
def test_switch_follows_the_oracle_state_machine(offload):
    gen = torch.Generator().manual_seed(41 + offload)
    rng = np.random.default_rng(41 + offload)
    th_h, t0_h = _inputs(gen)
    th = [x.to(DEV) for x in th_h]
    out = [torch.full((n,), 3.0, dtype=torch.bfloat16, device=DEV) for n in SIZES]
    keeps = [0.5, 0.0, 1.0, 0.5, 0.5, 0.5]
    params = [dict(s=1.0, keep=k, sigma=0.0, rescale=0, noise_kind=0) for k in keeps]
    th_np = [x.numpy() for x in th_h]
    t0_bits = [x.view(torch.int16).numpy().view(np.uint16) for x in t0_h]
    sw = oracle.StorageSwitch(th_np, t0_bits, offload=offload)
    if offload:
        hosts = [x.pin_memory() for x in t0_h]
        plan = smat.Plan(th, out, None, offload=True, theta0_hosts=hosts,
                         dtypes=(smat.SMAT_BF16, smat.SMAT_BF16, smat.SMAT_BF16))
    else:
        plan = smat.Plan(th, out, [x.to(DEV) for x in t0_h])
    lib = smat.lib()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    calls = {"simulate": 0, "to_simulated": 0, "to_expert": 0, "bad_target": 0, "bad_step": 0}
    errors = 0
    with plan:
        plan.set_params(params)
        for k in range(OPS):
            op = rng.choice(list(calls), p=[0.35, 0.3, 0.25, 0.05, 0.05])
            calls[op] += 1
            if op in ("simulate", "bad_step"):
                step = int(rng.integers(0, 1 << 30)) if op == "simulate" else int(rng.integers(1 << 30, 1 << 32))
                got = lib.smat_simulate_multi(plan._plan, SEED, step, stream)
                try:
                    want_out = [oracle.simulate(th_np[i], t0_bits[i], "bf16", "bf16", params[i], SEED, step, i)
                                for i in range(len(SIZES))]
                except ValueError:
                    want = _lib.SMAT_ERR_INVALID
                else:
                    try:
                        sw.simulate(want_out)
                        want = _lib.SMAT_OK
                    except oracle.StateError:
                        want = _lib.SMAT_ERR_STATE
            else:
                to = {"to_simulated": smat.SMAT_SIMULATED, "to_expert": smat.SMAT_EXPERT, "bad_target": 5}[op]
                got = lib.smat_switch_storage(plan._plan, to, stream)
                try:
                    sw.switch(to)
                    want = _lib.SMAT_OK
                except oracle.StateError:
                    want = _lib.SMAT_ERR_STATE
                except ValueError:
                    want = _lib.SMAT_ERR_INVALID
            what = f"call {k}: {op}"
            assert got == want, f"{what}: status {got}, oracle {want} ({lib.smat_last_error().decode()})"
            errors += got != 0
            assert plan.state == sw.state, what
            host_ptrs, dev_table = plan.active_ptrs()
            expect = [t.data_ptr() for t in (out if sw.state == oracle.SIMULATED else th)]
            assert host_ptrs == expect, what
            torch.cuda.synchronize()
            off = dev_table - plan.workspace.data_ptr()
            assert plan.workspace[off:off + 8 * len(SIZES)].cpu().view(torch.int64).tolist() == expect, what
            active = sw.active()
            for i in range(len(SIZES)):
                dev_active = out[i] if sw.state == oracle.SIMULATED else th[i]
                np.testing.assert_array_equal(_bits(dev_active), _np_bits(active[i]), err_msg=f"{what}, tensor {i}")
                if sw.buffer[i] is not None:
                    np.testing.assert_array_equal(_bits(out[i]), _np_bits(sw.buffer[i]),
                                                  err_msg=f"{what}, buffer of tensor {i}")
                np.testing.assert_array_equal(_bits(th[i]), th_np[i].view(np.uint32), err_msg=f"{what}, expert {i}")
    # the sequence exercised every kind of call, the misuse among them
    assert all(v > 0 for v in calls.values()), calls
    assert errors >= 20, errors
