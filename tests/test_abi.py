"""The C ABI library loads on the CPU, exports every function include/smat.h declares, and the
Python binding's structs match the C layout.  Only host-side argument checks are called here:
they return before any HIP call, so no GPU is needed."""
import ctypes
import os
import re
import shutil
import subprocess

import pytest

import paper_2609_33437_amd as smat
from paper_2609_33437_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "smat.h")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:smat_status|const char\*)\s+(smat_[a-z_]+)\(", text, re.M)))


def test_header_declares_the_binding_exports():
    assert _declared() == sorted(_lib.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(_lib.LIB_PATH)
    for name in _declared():
        assert hasattr(lib, name), name
    res = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True, text=True)
    if res.returncode == 0:
        exported = set(re.findall(r" T (smat_[a-z_]+)$", res.stdout, re.M))
        assert exported == set(_declared())


def test_struct_layout_matches_c(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None or not os.path.exists("/opt/rocm/include/hip/hip_runtime_api.h"):
        pytest.skip("gcc or HIP headers missing")
    src = tmp_path / "layout.c"
    src.write_text("""
#include <stdio.h>
#include <stddef.h>
#include "smat.h"
int main(void) {
  printf("%zu %zu %zu %zu %zu %zu %zu\\n", sizeof(smat_op_params), sizeof(smat_rng_key), sizeof(smat_tensor_desc),
         sizeof(smat_adamw_params), sizeof(smat_adam_state), sizeof(smat_merge_term), sizeof(smat_merge_desc));
  printf("%zu %zu %zu\\n", offsetof(smat_merge_term, seed), offsetof(smat_merge_desc, n),
         offsetof(smat_merge_desc, elem_offset));
  printf("%zu %zu %zu %zu\\n", offsetof(smat_tensor_desc, n), offsetof(smat_tensor_desc, tensor_id),
         offsetof(smat_tensor_desc, elem_offset), offsetof(smat_rng_key, elem_offset));
  printf("%zu %zu %zu\\n", sizeof(smat_step_state), offsetof(smat_step_state, step), offsetof(smat_step_state, scale));
  printf("%zu %zu\\n", sizeof(smat_adam_step_state), offsetof(smat_adam_step_state, step));
  return 0;
}
""")
    exe = tmp_path / "layout"
    subprocess.run([gcc, "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
                    str(src), "-o", str(exe)], check=True, capture_output=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split()
    want = [ctypes.sizeof(_lib.smat_op_params), ctypes.sizeof(_lib.smat_rng_key), ctypes.sizeof(_lib.smat_tensor_desc),
            ctypes.sizeof(_lib.smat_adamw_params), ctypes.sizeof(_lib.smat_adam_state),
            ctypes.sizeof(_lib.smat_merge_term), ctypes.sizeof(_lib.smat_merge_desc),
            _lib.smat_merge_term.seed.offset, _lib.smat_merge_desc.n.offset, _lib.smat_merge_desc.elem_offset.offset,
            _lib.smat_tensor_desc.n.offset, _lib.smat_tensor_desc.tensor_id.offset,
            _lib.smat_tensor_desc.elem_offset.offset, _lib.smat_rng_key.elem_offset.offset]
    # smat_step_state and smat_adam_step_state as StepState and AdamStepState pack them
    want += [16, 8, 12, 8, 4]
    assert [int(x) for x in out] == want


def _status(fn, *args):
    return fn(*args)


@pytest.mark.parametrize("bad", [dict(keep=1.5), dict(keep=-0.5), dict(sigma=-1.0), dict(sigma=float("inf")),
                                 dict(s=float("nan")), dict(noise_kind=9)])
def test_invalid_params_rejected_before_launch(bad):
    lib = smat.lib()
    p = _lib.op_params(dict(dict(s=0.5, keep=0.5, sigma=1e-3), **bad))
    key = _lib.rng_key(0, 0)
    st = lib.smat_simulate(ctypes.c_void_p(16), ctypes.c_void_p(4096), 1, ctypes.c_void_p(8192), 1, 4, p, key, None)
    assert st == _lib.SMAT_ERR_INVALID
    assert lib.smat_last_error().decode()


def test_argument_errors_without_gpu():
    lib = smat.lib()
    ok = _lib.op_params(dict(s=0.5, keep=0.5, sigma=1e-3))
    key = _lib.rng_key(0, 0)
    P = ctypes.c_void_p
    # dtype, negative size, null pointers, step range, aliasing
    assert lib.smat_simulate(P(16), P(4096), 7, P(8192), 1, 4, ok, key, None) == _lib.SMAT_ERR_DTYPE
    assert lib.smat_simulate(P(16), P(4096), 1, P(8192), 1, -1, ok, key, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_simulate(None, P(4096), 1, P(8192), 1, 4, ok, key, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_simulate(P(16), P(4096), 1, P(8192), 1, 4, ok, _lib.rng_key(0, 1 << 30), None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_simulate(P(4096), P(65536), 1, P(4096), 1, 4, ok, key, None) == _lib.SMAT_ERR_INVALID  # out == theta
    assert lib.smat_simulate(P(4096), P(65536), 1, P(65538), 1, 4, ok, key, None) == _lib.SMAT_ERR_INVALID  # partial overlap
    assert lib.smat_simulate(P(4096), P(65536), 0, P(65536), 1, 4, ok, key, None) == _lib.SMAT_ERR_INVALID  # in place, dtypes differ
    assert lib.smat_backward_accum(P(4096), 1, P(4100), 4, ok, 1.0, key, None) == _lib.SMAT_ERR_INVALID      # overlap
    assert lib.smat_backward_accum(P(4096), 1, P(65536), 4, ok, float("nan"), key, None) == _lib.SMAT_ERR_INVALID
    # n == 0 is a no-op even with null pointers
    assert lib.smat_simulate(None, None, 1, None, 1, 0, ok, key, None) == _lib.SMAT_OK


def _desc(theta, out, t0, gs, gt, n, tid, off=0, host=None):
    d = _lib.smat_tensor_desc()
    d.theta, d.out, d.theta0, d.grad_sim, d.grad_theta = theta, out, t0, gs, gt
    d.theta0_host = host
    d.n, d.tensor_id, d.elem_offset = n, tid, off
    return d


def test_plan_create_validation_without_gpu():
    lib = smat.lib()
    A = 1 << 20

    def plan(descs, offload=0, dts=(1, 1, 1)):
        arr = (_lib.smat_tensor_desc * len(descs))(*descs)
        p = ctypes.c_void_p()
        st = lib.smat_plan_create(arr, len(descs), dts[0], dts[1], dts[2], offload, ctypes.byref(p))
        if st == _lib.SMAT_OK:
            nb = ctypes.c_size_t()
            assert lib.smat_plan_workspace_bytes(p, ctypes.byref(nb)) == 0 and nb.value % 256 == 0
            s = ctypes.c_int32(-1)
            assert lib.smat_plan_state(p, ctypes.byref(s)) == 0 and s.value == _lib.SMAT_EXPERT
            assert lib.smat_plan_destroy(p) == 0
        return st

    good = [_desc(1 * A, 2 * A, 3 * A, 4 * A, 5 * A, 1000, 0), _desc(6 * A, 7 * A, 8 * A, 9 * A, 10 * A, 5, 1)]
    assert plan(good) == _lib.SMAT_OK
    # shards of one tensor may share a tensor id when their element ranges are disjoint
    shards = [_desc(1 * A, 2 * A, 3 * A, 4 * A, 5 * A, 1000, 7, 0), _desc(6 * A, 7 * A, 8 * A, 9 * A, 10 * A, 5, 7, 1000)]
    assert plan(shards) == _lib.SMAT_OK
    overlapping = [_desc(1 * A, 2 * A, 3 * A, 4 * A, 5 * A, 1000, 7, 0), _desc(6 * A, 7 * A, 8 * A, 9 * A, 10 * A, 5, 7, 999)]
    assert plan(overlapping) == _lib.SMAT_ERR_INVALID
    assert plan([_desc(1 * A, 1 * A, 3 * A, None, None, 10, 0)]) == _lib.SMAT_ERR_INVALID        # out over theta
    assert plan([_desc(1 * A, 2 * A, 3 * A, 4 * A, None, 10, 0)]) == _lib.SMAT_OK                # grad_sim only
    mixed = [_desc(1 * A, 2 * A, 3 * A, 4 * A, 5 * A, 10, 0), _desc(6 * A, 7 * A, 8 * A, None, None, 10, 1)]
    assert plan(mixed) == _lib.SMAT_ERR_INVALID                                                   # some tensors only
    assert plan([_desc(1 * A, 2 * A, 3 * A, 1 * A + 8, None, 10, 0)]) == _lib.SMAT_ERR_INVALID   # grad over theta
    assert plan(good, dts=(1, 1, 5)) == _lib.SMAT_ERR_DTYPE
    assert plan(good, offload=1) == _lib.SMAT_ERR_INVALID                                         # no host copy
    assert plan([_desc(1 * A, 2 * A, None, None, None, 10, 0, 0, 11 * A)], offload=1) == _lib.SMAT_OK
    assert plan([_desc(1 * A, 2 * A, None, None, None, 10, 0, 0, 11 * A)], offload=1, dts=(0, 1, 1)) == _lib.SMAT_ERR_INVALID
    # a plan without gradient pointers is valid for simulate-only use
    assert plan([_desc(1 * A, 2 * A, 3 * A, None, None, 10, 0)]) == _lib.SMAT_OK
    # more tensors than the kernels address with 32-bit record offsets: refused on the count alone,
    # before any descriptor is read (the array holds one)
    one = (_lib.smat_tensor_desc * 1)(good[0])
    p = ctypes.c_void_p()
    assert lib.smat_plan_create(one, (1 << 26) + 1, 1, 1, 1, 0, ctypes.byref(p)) == _lib.SMAT_ERR_INVALID
    assert b"at most" in lib.smat_last_error()
    # calls on an unbound plan fail with a state error and never launch
    arr = (_lib.smat_tensor_desc * 2)(*good)
    p = ctypes.c_void_p()
    assert lib.smat_plan_create(arr, 2, 1, 1, 1, 0, ctypes.byref(p)) == 0
    assert lib.smat_simulate_multi(p, 0, 0, None) == _lib.SMAT_ERR_STATE
    assert lib.smat_switch_storage(p, 1, None) == _lib.SMAT_ERR_STATE
    grads = (ctypes.c_void_p * 2)(ctypes.c_void_p(11 * A), ctypes.c_void_p(12 * A))
    assert lib.smat_plan_set_grads(p, grads, None, None) == _lib.SMAT_ERR_STATE        # no workspace yet
    assert lib.smat_plan_set_grads(p, None, None, None) == _lib.SMAT_ERR_INVALID       # nothing to set
    assert lib.smat_switch_storage(p, 5, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_plan_destroy(p) == 0
    assert lib.smat_plan_destroy(None) == 0


def test_device_driven_calls_without_gpu():
    """The device-driven list calls check their arguments and the plan's state on the host and
    return before any HIP call: null or misaligned state, offload plans, unbound plans."""
    lib = smat.lib()
    lib.smat_last_error.restype = ctypes.c_char_p
    A = 1 << 20
    state = ctypes.c_void_p(64 * A)
    arr = (_lib.smat_tensor_desc * 1)(_desc(1 * A, 2 * A, 3 * A, 4 * A, 5 * A, 1000, 0))
    p = ctypes.c_void_p()
    assert lib.smat_plan_create(arr, 1, 1, 1, 1, 0, ctypes.byref(p)) == 0
    assert lib.smat_simulate_multi_dev(None, state, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_simulate_multi_dev(p, None, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_simulate_multi_dev(p, ctypes.c_void_p(64 * A + 8), None) == _lib.SMAT_ERR_INVALID
    assert b"16-byte aligned" in lib.smat_last_error()
    assert lib.smat_simulate_multi_dev(p, state, None) == _lib.SMAT_ERR_STATE           # no workspace
    assert lib.smat_backward_multi_dev(p, None, 1.0, 1, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_backward_multi_dev(p, state, 1.0, 1, None) == _lib.SMAT_ERR_STATE    # no workspace
    hp = _lib.adamw_params(dict(lr=0.0, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, step=1))
    adam = ctypes.c_void_p(65 * A)
    sq = ctypes.c_void_p(66 * A)
    assert lib.smat_adamw_fused_multi_dev(p, None, adam, hp, 1.0, 0, None, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_adamw_fused_multi_dev(p, state, adam, hp, 1.0, 0, None, None) == _lib.SMAT_ERR_STATE
    assert lib.smat_grad_norm_multi_dev(p, state, 1.0, 0, 1.0, sq, None, None) == _lib.SMAT_ERR_STATE
    assert lib.smat_grad_norm_multi_dev(None, state, 1.0, 0, 1.0, sq, None, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_plan_destroy(p) == 0
    assert lib.smat_step_state_advance(None, 1, 0.2, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_step_state_advance(ctypes.c_void_p(64 * A + 8), 1, 0.2, None) == _lib.SMAT_ERR_INVALID
    for bad in (-0.1, 1.5, float("nan")):
        assert lib.smat_step_state_advance(state, 1, bad, None) == _lib.SMAT_ERR_INVALID
    arr = (_lib.smat_tensor_desc * 1)(_desc(1 * A, 2 * A, None, 4 * A, 5 * A, 1000, 0, 0, 11 * A))
    assert lib.smat_plan_create(arr, 1, 1, 1, 1, 1, ctypes.byref(p)) == 0
    assert lib.smat_simulate_multi_dev(p, state, None) == _lib.SMAT_ERR_STATE
    assert b"offload" in lib.smat_last_error()
    assert lib.smat_backward_multi_dev(p, state, 1.0, 0, None) == _lib.SMAT_ERR_STATE
    assert lib.smat_plan_destroy(p) == 0


def test_clear_grads_without_gpu():
    """Clearing is host-side: it validates `which`, and afterwards the operations that read a cleared
    kind are state errors whatever else is missing."""
    lib = smat.lib()
    A = 1 << 20
    arr = (_lib.smat_tensor_desc * 1)(_desc(1 * A, 2 * A, 3 * A, 4 * A, 5 * A, 1000, 0))
    p = ctypes.c_void_p()
    assert lib.smat_plan_create(arr, 1, 1, 1, 1, 0, ctypes.byref(p)) == 0
    assert lib.smat_plan_clear_grads(None, 3) == _lib.SMAT_ERR_INVALID
    for bad in (0, 4, -1):
        assert lib.smat_plan_clear_grads(p, bad) == _lib.SMAT_ERR_INVALID
    assert lib.smat_plan_clear_grads(p, 2) == _lib.SMAT_OK
    lib.smat_last_error.restype = ctypes.c_char_p
    assert lib.smat_backward_multi(p, 0, 0, 1.0, 0, None) == _lib.SMAT_ERR_STATE        # grad_theta gone
    assert b"gradient arrays not set" in lib.smat_last_error()
    assert lib.smat_grad_norm_multi(p, 0, 0, 1.0, 1, 1.0, ctypes.c_void_p(6 * A), None, None) == _lib.SMAT_ERR_STATE
    assert b"gradient arrays not set" in lib.smat_last_error()
    assert lib.smat_plan_clear_grads(p, 1) == _lib.SMAT_OK
    assert lib.smat_grad_norm_multi(p, 0, 0, 1.0, 0, 1.0, ctypes.c_void_p(6 * A), None, None) == _lib.SMAT_ERR_STATE
    assert b"gradient arrays not set" in lib.smat_last_error()
    assert lib.smat_plan_clear_grads(p, 3) == _lib.SMAT_OK                               # clearing twice is fine
    assert lib.smat_plan_destroy(p) == 0


@pytest.mark.parametrize("bad", [dict(beta1=1.0), dict(beta2=-0.5), dict(eps=0.0), dict(lr=-1.0), dict(step=0),
                                 dict(weight_decay=float("nan")), dict(grad_scale=float("inf"))])
def test_invalid_adamw_hyperparameters_rejected_before_launch(bad):
    lib = smat.lib()
    hp = _lib.adamw_params(dict(dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, step=1), **bad))
    p = _lib.op_params(dict(s=0.5, keep=0.5, sigma=0.0))
    P = ctypes.c_void_p
    st = lib.smat_adamw_fused(P(1 << 20), 1, None, P(2 << 20), P(3 << 20), P(4 << 20), 4, p, 1.0, hp,
                              _lib.rng_key(0, 0), None, None)
    assert st == _lib.SMAT_ERR_INVALID


def test_adamw_overlap_rejected_without_gpu():
    lib = smat.lib()
    hp = _lib.adamw_params(dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, step=1))
    p = _lib.op_params(dict(s=0.5, keep=0.5, sigma=0.0))
    P = ctypes.c_void_p
    # exp_avg overlaps theta
    st = lib.smat_adamw_fused(P(1 << 20), 1, None, P(2 << 20), P((2 << 20) + 8), P(4 << 20), 4, p, 1.0, hp,
                              _lib.rng_key(0, 0), None, None)
    assert st == _lib.SMAT_ERR_INVALID


def test_grad_norm_argument_errors_without_gpu():
    lib = smat.lib()
    A = 1 << 20
    P = ctypes.c_void_p
    arr = (_lib.smat_tensor_desc * 1)(_desc(1 * A, 2 * A, 3 * A, 4 * A, 5 * A, 1000, 0))
    plan = P()
    assert lib.smat_plan_create(arr, 1, 1, 1, 1, 0, ctypes.byref(plan)) == 0
    out = P(6 * A)
    assert lib.smat_grad_norm_multi(None, 0, 0, 1.0, 0, 1.0, out, None, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_grad_norm_multi(plan, 0, 0, 1.0, 0, 1.0, None, None, None) == _lib.SMAT_ERR_INVALID   # no output
    for bad in (0.0, -1.0, float("nan"), float("inf")):
        assert lib.smat_grad_norm_multi(plan, 0, 0, 1.0, 0, bad, None, out, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_grad_norm_multi(plan, 0, 0, float("inf"), 0, 1.0, out, None, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_grad_norm_multi(plan, 0, 0, 1.0, 2, 1.0, out, None, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_grad_norm_multi(plan, 0, 1 << 30, 1.0, 0, 1.0, out, None, None) == _lib.SMAT_ERR_INVALID
    # a valid call on a plan without workspace is a state error and launches nothing
    assert lib.smat_grad_norm_multi(plan, 0, 0, 1.0, 0, 1.0, out, None, None) == _lib.SMAT_ERR_STATE
    assert lib.smat_plan_destroy(plan) == 0
    # a plan without gradient arrays has no norm to take until smat_plan_set_grads supplies them
    arr = (_lib.smat_tensor_desc * 1)(_desc(1 * A, 2 * A, 3 * A, None, None, 1000, 0))
    assert lib.smat_plan_create(arr, 1, 1, 1, 1, 0, ctypes.byref(plan)) == 0
    assert lib.smat_grad_norm_multi(plan, 0, 0, 1.0, 0, 1.0, out, None, None) == _lib.SMAT_ERR_STATE
    assert lib.smat_plan_destroy(plan) == 0


def test_merge_argument_errors_without_gpu():
    lib = smat.lib()
    P = ctypes.c_void_p
    A = 1 << 20
    T = _lib.smat_merge_term
    good = (T * 2)(T(0.3, 0.7, 1, 0, 5), T(0.3, 1.0, 1, 0, 6))
    ex = (P * 2)(P(1 * A), P(2 * A))
    assert lib.smat_merge(ex, 2, 1, P(3 * A), 1, P(4 * A), 1, 0, good, 0, 0, None) == _lib.SMAT_OK      # n == 0
    assert lib.smat_merge(ex, 0, 1, P(3 * A), 1, P(4 * A), 1, 4, good, 0, 0, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_merge(ex, 17, 1, P(3 * A), 1, P(4 * A), 1, 4, good, 0, 0, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_merge(ex, 2, 9, P(3 * A), 1, P(4 * A), 1, 4, good, 0, 0, None) == _lib.SMAT_ERR_DTYPE
    for bad in (T(float("nan"), 1.0, 1, 0, 0), T(0.3, 1.5, 1, 0, 0), T(0.3, -0.1, 1, 0, 0), T(0.3, 0.5, 1, 1 << 30, 0)):
        terms = (T * 2)(good[0], bad)
        assert lib.smat_merge(ex, 2, 1, P(3 * A), 1, P(4 * A), 1, 4, terms, 0, 0, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_merge(ex, 2, 1, P(3 * A), 1, P(2 * A + 2), 1, 4, good, 0, 0, None) == _lib.SMAT_ERR_INVALID  # out over expert
    assert lib.smat_merge(ex, 2, 1, P(3 * A), 1, P(3 * A + 2), 1, 4, good, 0, 0, None) == _lib.SMAT_ERR_INVALID  # out over theta0
    assert lib.smat_merge(ex, 2, 1, P(3 * A), 0, P(3 * A), 1, 4, good, 0, 0, None) == _lib.SMAT_ERR_INVALID      # in place, dtypes differ
    nul = (P * 2)(P(1 * A), None)
    assert lib.smat_merge(nul, 2, 1, P(3 * A), 1, P(4 * A), 1, 4, good, 0, 0, None) == _lib.SMAT_ERR_INVALID


def test_merge_plan_validation_without_gpu():
    lib = smat.lib()
    P = ctypes.c_void_p
    A = 1 << 20
    D = _lib.smat_merge_desc

    def create(descs, ptrs, nexp=2, dts=(1, 1, 1)):
        arr = (D * len(descs))(*descs)
        ex = (P * len(ptrs))(*ptrs)
        p = P()
        st = lib.smat_merge_plan_create(arr, len(descs), ex, nexp, dts[0], dts[1], dts[2], ctypes.byref(p))
        if st == _lib.SMAT_OK:
            nb = ctypes.c_size_t()
            assert lib.smat_merge_plan_workspace_bytes(p, ctypes.byref(nb)) == 0 and nb.value % 256 == 0
            terms = (_lib.smat_merge_term * max(1, len(descs) * nexp))()
            assert lib.smat_merge_multi(p, terms, None) == _lib.SMAT_ERR_STATE      # no workspace: nothing launched
            assert lib.smat_merge_plan_destroy(p) == 0
        return st

    two = [D(P(1 * A), P(2 * A), 1000, 0, 0, 0), D(P(3 * A), P(4 * A), 10, 1, 0, 0)]
    ptrs = [P(5 * A), P(6 * A), P(7 * A), P(8 * A)]
    assert create(two, ptrs) == _lib.SMAT_OK
    assert create(two, ptrs, nexp=0) == _lib.SMAT_ERR_INVALID
    assert create(two, ptrs, dts=(1, 1, 4)) == _lib.SMAT_ERR_DTYPE
    assert create([D(P(1 * A), P(2 * A), 1000, 0, 1, 0)], ptrs[:2]) == _lib.SMAT_ERR_INVALID        # reserved != 0
    assert create([D(P(1 * A), P(5 * A + 8), 1000, 0, 0, 0)], ptrs[:2]) == _lib.SMAT_ERR_INVALID    # out over an expert
    assert create([D(P(1 * A), P(1 * A), 1000, 0, 0, 0)], ptrs[:2]) == _lib.SMAT_OK                 # in place over theta0
    overlapping = [D(P(1 * A), P(2 * A), 1000, 7, 0, 0), D(P(3 * A), P(4 * A), 10, 7, 0, 999)]
    assert create(overlapping, ptrs) == _lib.SMAT_ERR_INVALID
    shards = [D(P(1 * A), P(2 * A), 1000, 7, 0, 0), D(P(3 * A), P(4 * A), 10, 7, 0, 1000)]
    assert create(shards, ptrs) == _lib.SMAT_OK
    assert lib.smat_merge_plan_destroy(None) == 0


def test_stream_copy_argument_errors_without_gpu():
    lib = smat.lib()
    P = ctypes.c_void_p
    assert lib.smat_stream_copy(P(1 << 20), P(2 << 20), 0, None) == _lib.SMAT_OK               # nothing to copy
    assert lib.smat_stream_copy(None, P(2 << 20), 16, None) == _lib.SMAT_ERR_INVALID
    assert lib.smat_stream_copy(P((1 << 20) + 8), P(2 << 20), 16, None) == _lib.SMAT_ERR_INVALID  # misaligned
    assert lib.smat_stream_copy(P(1 << 20), P(2 << 20), 24, None) == _lib.SMAT_ERR_INVALID       # size
    assert lib.smat_stream_copy(P(1 << 20), P((1 << 20) + 16), 64, None) == _lib.SMAT_ERR_INVALID  # overlap


def test_scale_draw_matches_oracle_without_gpu():
    """smat_scale_draw is host code: the step's scale, bit for bit the oracle's draw, for many keys."""
    import numpy as np
    import oracle
    rng = np.random.default_rng(3)
    for _ in range(300):
        seed = int(rng.integers(0, 2 ** 63)) * 2 + int(rng.integers(0, 2))
        step = int(rng.integers(0, 2 ** 30))
        amin = float(rng.choice([0.0, 0.1, 0.2, float(rng.random()), 1.0]))
        assert smat.scale_draw(seed, step, amin) == oracle.scale_draw(seed, step, amin), (seed, step, amin)
    lib = smat.lib()
    out = ctypes.c_float()
    assert lib.smat_scale_draw(1, 2, 1.5, ctypes.byref(out)) == _lib.SMAT_ERR_INVALID
    assert lib.smat_scale_draw(1, 2, 0.5, None) == _lib.SMAT_ERR_INVALID
    # steps live in [0, 2^30), as in the host-driven calls and the oracle
    assert lib.smat_scale_draw(1, 2 ** 30 - 1, 0.5, ctypes.byref(out)) == _lib.SMAT_OK
    assert lib.smat_scale_draw(1, 2 ** 30, 0.5, ctypes.byref(out)) == _lib.SMAT_ERR_INVALID
    with pytest.raises(ValueError):
        oracle.scale_draw(1, 2 ** 30, 0.5)


def test_every_entry_point_survives_zero_arguments():
    """Every exported call, given null pointers, zero counts and zeroed records, returns a status
    (a no-op or an argument error) without touching memory or needing a GPU."""
    lib = smat.lib()
    statuses = {}
    for name in _lib.EXPORTS:
        if name == "smat_last_error":
            continue
        fn = getattr(lib, name)
        args = []
        for t in fn.argtypes:
            if isinstance(t, type) and issubclass(t, ctypes.Structure):
                args.append(t())
            elif t in (ctypes.c_float, ctypes.c_double):
                args.append(0.0)
            elif t in (ctypes.c_int32, ctypes.c_uint32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_size_t):
                args.append(0)
            else:
                args.append(None)
        statuses[name] = fn(*args)
    allowed = (_lib.SMAT_OK, _lib.SMAT_ERR_INVALID, _lib.SMAT_ERR_DTYPE, _lib.SMAT_ERR_STATE)
    assert all(st in allowed for st in statuses.values()), statuses
    # calls that take a plan or an output pointer refuse a null one
    for name, st in statuses.items():
        if "plan" in name and name not in ("smat_plan_destroy", "smat_merge_plan_destroy"):
            assert st == _lib.SMAT_ERR_INVALID, name
