"""ctypes binding of libsmat (argument marshalling only; every step runs in the HIP kernels).

The functions keep the C names.  Tensors are PyTorch tensors on the GPU (torch supplies device
memory and the HIP stream); scalars and parameter records are marshalled into the C structs of
include/smat.h.  There is no fallback: without the built library importing this module fails.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_float, c_int32, c_int64, c_size_t, c_uint32, c_uint64, c_void_p
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsmat.so")

SMAT_OK, SMAT_ERR_INVALID, SMAT_ERR_DTYPE, SMAT_ERR_STATE, SMAT_ERR_HIP = 0, 1, 2, 3, 4
SMAT_F32, SMAT_BF16 = 0, 1
SMAT_NOISE_GAUSSIAN, SMAT_NOISE_UNIFORM, SMAT_NOISE_LAPLACE = 0, 1, 2
SMAT_EXPERT, SMAT_SIMULATED = 0, 1

STATUS_NAMES = {0: "SMAT_OK", 1: "SMAT_ERR_INVALID", 2: "SMAT_ERR_DTYPE", 3: "SMAT_ERR_STATE", 4: "SMAT_ERR_HIP"}

EXPORTS = (
    "smat_simulate", "smat_backward_accum", "smat_debug_draws", "smat_plan_create", "smat_plan_workspace_bytes",
    "smat_plan_bind_workspace", "smat_plan_set_params", "smat_simulate_multi", "smat_backward_accum_multi",
    "smat_switch_storage", "smat_plan_state", "smat_plan_active_ptrs", "smat_plan_destroy", "smat_last_error",
    "smat_adamw_fused", "smat_plan_bind_adam_state", "smat_adamw_fused_multi", "smat_grad_norm_multi",
    "smat_merge", "smat_merge_plan_create", "smat_merge_plan_workspace_bytes", "smat_merge_plan_bind_workspace",
    "smat_merge_multi", "smat_merge_plan_destroy", "smat_plan_set_grads",
    "smat_stream_copy", "smat_backward_multi", "smat_plan_clear_grads", "smat_simulate_multi_dev",
    "smat_backward_multi_dev", "smat_adamw_fused_multi_dev", "smat_grad_norm_multi_dev", "smat_step_state_advance",
    "smat_scale_draw", "smat_simulate_multi_static",
)


class smat_op_params(ctypes.Structure):
    _fields_ = [("s", c_float), ("keep", c_float), ("sigma", c_float), ("rescale", c_int32), ("noise_kind", c_int32)]


# smat_op_params as a NumPy record, for lists of per-tensor parameters filled column by column
OP_PARAMS_DTYPE = np.dtype([("s", "<f4"), ("keep", "<f4"), ("sigma", "<f4"), ("rescale", "<i4"),
                            ("noise_kind", "<i4")], align=True)
assert OP_PARAMS_DTYPE.itemsize == ctypes.sizeof(smat_op_params)


def op_params_array(count: int, s, keep, sigma, rescale=1, noise_kind=0) -> np.ndarray:
    """`count` smat_op_params records in one array; each field is a scalar shared by all tensors or
    a sequence of `count` values.  Plan.set_params takes it without a per-tensor Python loop."""
    a = np.empty(count, dtype=OP_PARAMS_DTYPE)
    a["s"], a["keep"], a["sigma"], a["rescale"], a["noise_kind"] = s, keep, sigma, rescale, noise_kind
    return a


class smat_rng_key(ctypes.Structure):
    _fields_ = [("seed", c_uint64), ("step", c_uint32), ("tensor_id", c_uint32), ("elem_offset", c_uint64)]


class smat_tensor_desc(ctypes.Structure):
    _fields_ = [("theta", c_void_p), ("theta0", c_void_p), ("out", c_void_p), ("grad_sim", c_void_p),
                ("grad_theta", c_void_p), ("theta0_host", c_void_p), ("n", c_int64), ("tensor_id", c_uint32),
                ("reserved", c_uint32), ("elem_offset", c_uint64)]


class smat_adamw_params(ctypes.Structure):
    _fields_ = [("lr", c_float), ("beta1", c_float), ("beta2", c_float), ("eps", c_float),
                ("weight_decay", c_float), ("grad_scale", c_float), ("step", c_int32)]


class smat_adam_state(ctypes.Structure):
    _fields_ = [("exp_avg", c_void_p), ("exp_avg_sq", c_void_p)]


class smat_merge_term(ctypes.Structure):
    _fields_ = [("gamma", c_float), ("keep", c_float), ("rescale", c_int32), ("step", c_uint32), ("seed", c_uint64)]


class smat_merge_desc(ctypes.Structure):
    _fields_ = [("theta0", c_void_p), ("out", c_void_p), ("n", c_int64), ("tensor_id", c_uint32),
                ("reserved", c_uint32), ("elem_offset", c_uint64)]


class SmatError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build the HIP library first "
                          "(python -m paper_2609_33437_amd.build)")
    lib = ctypes.CDLL(path)
    P = c_void_p
    sig = {
        "smat_simulate": [P, P, c_int32, P, c_int32, c_int64, smat_op_params, smat_rng_key, P],
        "smat_backward_accum": [P, c_int32, P, c_int64, smat_op_params, c_float, smat_rng_key, P],
        "smat_debug_draws": [smat_rng_key, c_int64, smat_op_params, P, P, P, P, P],
        "smat_plan_create": [POINTER(smat_tensor_desc), c_int32, c_int32, c_int32, c_int32, c_int32, POINTER(P)],
        "smat_plan_workspace_bytes": [P, POINTER(c_size_t)],
        "smat_plan_bind_workspace": [P, P, c_size_t, P],
        "smat_plan_set_params": [P, POINTER(smat_op_params), P],
        "smat_simulate_multi": [P, c_uint64, c_uint32, P],
        "smat_backward_accum_multi": [P, c_uint64, c_uint32, c_float, P],
        "smat_switch_storage": [P, c_int32, P],
        "smat_plan_state": [P, POINTER(c_int32)],
        "smat_plan_active_ptrs": [P, POINTER(P), POINTER(P)],
        "smat_plan_destroy": [P],
        "smat_adamw_fused": [P, c_int32, P, P, P, P, c_int64, smat_op_params, c_float, smat_adamw_params,
                             smat_rng_key, P, P],
        "smat_plan_bind_adam_state": [P, POINTER(smat_adam_state), P],
        "smat_adamw_fused_multi": [P, c_uint64, c_uint32, c_float, smat_adamw_params, c_int32, P, P],
        "smat_grad_norm_multi": [P, c_uint64, c_uint32, c_float, c_int32, c_float, P, P, P],
        "smat_merge": [POINTER(P), c_int32, c_int32, P, c_int32, P, c_int32, c_int64, POINTER(smat_merge_term),
                       c_uint32, c_uint64, P],
        "smat_merge_plan_create": [POINTER(smat_merge_desc), c_int32, POINTER(P), c_int32, c_int32, c_int32, c_int32,
                                   POINTER(P)],
        "smat_merge_plan_workspace_bytes": [P, POINTER(c_size_t)],
        "smat_merge_plan_bind_workspace": [P, P, c_size_t, P],
        "smat_merge_multi": [P, POINTER(smat_merge_term), P],
        "smat_merge_plan_destroy": [P],
        "smat_plan_set_grads": [P, POINTER(P), POINTER(P), P],
        "smat_stream_copy": [P, P, c_uint64, P],
        "smat_backward_multi": [P, c_uint64, c_uint32, c_float, c_int32, P],
        "smat_plan_clear_grads": [P, c_int32],
        "smat_simulate_multi_dev": [P, P, P],
        "smat_backward_multi_dev": [P, P, c_float, c_int32, P],
        "smat_adamw_fused_multi_dev": [P, P, P, smat_adamw_params, c_float, c_int32, P, P],
        "smat_grad_norm_multi_dev": [P, P, c_float, c_int32, c_float, P, P, P],
        "smat_step_state_advance": [P, c_uint32, c_float, P],
        "smat_scale_draw": [c_uint64, c_uint32, c_float, POINTER(c_float)],
        "smat_simulate_multi_static": [POINTER(smat_tensor_desc), c_int32, c_int32, c_int32, POINTER(smat_op_params),
                                       c_uint64, c_uint32, P],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = c_int32
    lib.smat_last_error.argtypes = []
    lib.smat_last_error.restype = c_char_p
    return lib


_LIB: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    global _LIB
    if _LIB is None:
        _LIB = load_library()
    return _LIB


def _check(status: int) -> None:
    if status != SMAT_OK:
        raise SmatError(status, lib().smat_last_error().decode())


# ------------------------------------------------------------------ marshalling helpers
def _torch():
    import torch
    return torch


def dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return SMAT_F32
    if t.dtype == torch.bfloat16:
        return SMAT_BF16
    raise SmatError(SMAT_ERR_DTYPE, f"unsupported tensor dtype {t.dtype}")


def _stream_handle(stream) -> c_void_p:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return c_void_p(s.cuda_stream)


def _dev_ptr(t, what: str):
    if t is None:
        return None
    if not t.is_cuda:
        raise SmatError(SMAT_ERR_INVALID, f"{what} must be a GPU tensor")
    if not t.is_contiguous():
        raise SmatError(SMAT_ERR_INVALID, f"{what} must be contiguous")
    return c_void_p(t.data_ptr()) if t.numel() else None


def _scalar_ptr(t, what: str, dtype: str):
    """Device pointer of a one-element GPU tensor of the given dtype (None passes NULL)."""
    if t is None:
        return None
    if str(t.dtype) != f"torch.{dtype}" or t.numel() != 1:
        raise SmatError(SMAT_ERR_INVALID, f"{what} must be a one-element {dtype} tensor")
    return _dev_ptr(t, what)


def scale_draw(seed: int, step: int, alpha_min: float) -> float:
    """The step's shared scale alpha ~ U[alpha_min, 1] as a function of (seed, step): the value
    smat_step_state_advance writes on the GPU, computed on the host (smat_scale_draw)."""
    if not (0 <= int(seed) < 2 ** 64 and 0 <= int(step) < 2 ** 32):
        raise SmatError(SMAT_ERR_INVALID, "seed must fit 64 bits and step 32 bits (the library takes steps < 2^30)")
    out = c_float()
    _check(lib().smat_scale_draw(int(seed), int(step), float(alpha_min), ctypes.byref(out)))
    return out.value


class StepState:
    """The 16 bytes that the device-driven list calls read when their kernels run, in GPU memory:
    seed (uint64), step (uint32), scale (float32), the layout of smat_step_state.

    set() writes all three from the host (between graph replays); seed_view, step_view and
    scale_view are one-element views of the same bytes that torch ops, captured into the same graph,
    can update in place (for example step_view.add_(1), or scale_view.copy_ of a sampled scale)."""

    def __init__(self, seed: int = 0, step: int = 0, scale: float = 1.0, device=None):
        torch = _torch()
        self.tensor = torch.zeros(4, dtype=torch.int32, device=device if device is not None else "cuda")
        self.set(seed, step, scale)

    def set(self, seed: int, step: int, scale: float) -> None:
        import numpy as np
        rec = np.zeros(1, dtype=[("seed", "<u8"), ("step", "<u4"), ("scale", "<f4")])
        rec["seed"], rec["step"], rec["scale"] = int(seed), int(step), float(scale)
        self.tensor.copy_(_torch().from_numpy(rec.view(np.int32).copy()))

    def advance(self, alpha_min: float, increment: int = 1, stream=None) -> None:
        """smat_step_state_advance on the GPU: step += increment, then the scale of that step
        drawn from (seed, step) as alpha ~ U[alpha_min, 1].  Capturable."""
        _check(lib().smat_step_state_advance(_dev_ptr(self.tensor, "step state"), int(increment) & 0xFFFFFFFF,
                                             float(alpha_min), _stream_handle(stream)))

    @property
    def seed_view(self):
        return self.tensor[0:2].view(_torch().int64)

    @property
    def step_view(self):
        return self.tensor[2:3]

    @property
    def scale_view(self):
        return self.tensor[3:4].view(_torch().float32)


class AdamStepState:
    """The optimizer's per-step values for the device-driven fused optimizer step, in GPU memory:
    lr (float32) and the step count (uint32), the layout of smat_adam_step_state.  lr_view and
    step_view are one-element views that captured torch ops can update in place."""

    def __init__(self, lr: float = 0.0, step: int = 1, device=None):
        torch = _torch()
        self.tensor = torch.zeros(2, dtype=torch.int32, device=device if device is not None else "cuda")
        self.set(lr, step)

    def set(self, lr: float, step: int) -> None:
        import numpy as np
        rec = np.zeros(1, dtype=[("lr", "<f4"), ("step", "<u4")])
        rec["lr"], rec["step"] = float(lr), int(step)
        self.tensor.copy_(_torch().from_numpy(rec.view(np.int32).copy()))

    @property
    def lr_view(self):
        return self.tensor[0:1].view(_torch().float32)

    @property
    def step_view(self):
        return self.tensor[1:2]


def _state_ptr(state, cls=StepState, nbytes: int = 16, what: str = "step state"):
    """Device pointer of a StepState (AdamStepState), or of a contiguous GPU tensor of its size."""
    t = state.tensor if isinstance(state, cls) else state
    if t is None or t.numel() * t.element_size() != nbytes:
        raise SmatError(SMAT_ERR_INVALID, f"{what} must be a {cls.__name__} or a {nbytes}-byte GPU tensor")
    return _dev_ptr(t, what)


def _expect(t, n: int, code: int, what: str) -> None:
    """The C ABI sees only pointers and element counts, so the binding checks that each array holds
    exactly n elements of the dtype the launch assumes (a shorter or narrower array would be
    overrun by the kernel)."""
    if t is None:
        return
    if t.numel() != n:
        raise SmatError(SMAT_ERR_INVALID, f"{what} holds {t.numel()} elements, expected {n}")
    if dtype_code(t) != code:
        raise SmatError(SMAT_ERR_DTYPE, f"{what} has dtype {t.dtype}, expected {'float32' if code == SMAT_F32 else 'bfloat16'}")


def op_params(p) -> smat_op_params:
    """dict(s, keep, sigma, rescale=1, noise_kind=0) or an smat_op_params -> smat_op_params."""
    if isinstance(p, smat_op_params):
        return p
    return smat_op_params(float(p["s"]), float(p["keep"]), float(p["sigma"]), int(p.get("rescale", 1)),
                          int(p.get("noise_kind", SMAT_NOISE_GAUSSIAN)))


def rng_key(seed: int, step: int, tensor_id: int = 0, elem_offset: int = 0) -> smat_rng_key:
    return smat_rng_key(int(seed), int(step), int(tensor_id), int(elem_offset))


def adamw_params(hp) -> smat_adamw_params:
    """dict(lr, beta1, beta2, eps, weight_decay, grad_scale=1, step) or an smat_adamw_params."""
    if isinstance(hp, smat_adamw_params):
        return hp
    return smat_adamw_params(float(hp["lr"]), float(hp["beta1"]), float(hp["beta2"]), float(hp["eps"]),
                             float(hp["weight_decay"]), float(hp.get("grad_scale", 1.0)), int(hp["step"]))


# ------------------------------------------------------------------ single tensor
def smat_simulate(theta, theta0, out, params, seed: int, step: int, tensor_id: int = 0, elem_offset: int = 0,
                  stream=None) -> None:
    """theta~ of one flat tensor into `out` (see include/smat.h)."""
    n = theta.numel()
    if theta0.numel() != n or out.numel() != n:
        raise SmatError(SMAT_ERR_INVALID, "theta, theta0 and out differ in size")
    _expect(theta, n, SMAT_F32, "theta")
    _check(lib().smat_simulate(_dev_ptr(theta, "theta"), _dev_ptr(theta0, "theta0"), dtype_code(theta0),
                               _dev_ptr(out, "out"), dtype_code(out), n, op_params(params),
                               rng_key(seed, step, tensor_id, elem_offset), _stream_handle(stream)))


def smat_backward_accum(grad_sim, grad_theta, params, lam: float, seed: int, step: int, tensor_id: int = 0,
                        elem_offset: int = 0, stream=None) -> None:
    """grad_theta += lam * t * m * grad_sim in place (see include/smat.h)."""
    n = grad_theta.numel()
    if grad_sim.numel() != n:
        raise SmatError(SMAT_ERR_INVALID, "grad_sim and grad_theta differ in size")
    _expect(grad_theta, n, SMAT_F32, "grad_theta")
    _check(lib().smat_backward_accum(_dev_ptr(grad_sim, "grad_sim"), dtype_code(grad_sim),
                                     _dev_ptr(grad_theta, "grad_theta"), n, op_params(params), float(lam),
                                     rng_key(seed, step, tensor_id, elem_offset), _stream_handle(stream)))


def smat_debug_draws(n: int, params, seed: int, step: int, tensor_id: int = 0, elem_offset: int = 0,
                     mask_words=None, noise_words=None, kept=None, z=None, stream=None) -> None:
    """Raw per-element draws into the given GPU tensors (uint32 viewed as int32, uint8, fp32)."""
    torch = _torch()
    for name, t, size in (("mask_words", mask_words, 4), ("noise_words", noise_words, 4), ("kept", kept, 1),
                          ("z", z, 4)):
        if t is not None and (t.numel() != n or t.element_size() != size):
            raise SmatError(SMAT_ERR_INVALID, f"{name} must hold n elements of {size} byte(s)")
    if z is not None and z.dtype != torch.float32:
        raise SmatError(SMAT_ERR_DTYPE, "z must be float32")
    _check(lib().smat_debug_draws(rng_key(seed, step, tensor_id, elem_offset), int(n), op_params(params),
                                  _dev_ptr(mask_words, "mask_words"), _dev_ptr(noise_words, "noise_words"),
                                  _dev_ptr(kept, "kept"), _dev_ptr(z, "z"), _stream_handle(stream)))


def smat_adamw_fused(grad_sim, theta, exp_avg, exp_avg_sq, params, lam: float, hp, seed: int, step: int,
                     tensor_id: int = 0, elem_offset: int = 0, grad_acc=None, grad_scale_dev=None,
                     stream=None) -> None:
    """One AdamW step of theta from grad_acc + lam * t * m * grad_sim, in place (see include/smat.h).
    grad_scale_dev: optional one-element fp32 GPU tensor multiplying the gradient (read on the GPU)."""
    n = theta.numel()
    for name, t in (("grad_sim", grad_sim), ("exp_avg", exp_avg), ("exp_avg_sq", exp_avg_sq), ("grad_acc", grad_acc)):
        if t is not None and t.numel() != n:
            raise SmatError(SMAT_ERR_INVALID, f"{name} differs in size from theta")
    for name, t in (("theta", theta), ("exp_avg", exp_avg), ("exp_avg_sq", exp_avg_sq), ("grad_acc", grad_acc)):
        _expect(t, n, SMAT_F32, name)
    _check(lib().smat_adamw_fused(_dev_ptr(grad_sim, "grad_sim"), dtype_code(grad_sim), _dev_ptr(grad_acc, "grad_acc"),
                                  _dev_ptr(theta, "theta"), _dev_ptr(exp_avg, "exp_avg"),
                                  _dev_ptr(exp_avg_sq, "exp_avg_sq"), n, op_params(params), float(lam),
                                  adamw_params(hp), rng_key(seed, step, tensor_id, elem_offset),
                                  _scalar_ptr(grad_scale_dev, "grad_scale_dev", "float32"), _stream_handle(stream)))


# ------------------------------------------------------------------ tensor-list plans
class Plan:
    """A tensor list bound to libsmat (smat_plan_* calls); holds references to its tensors."""

    def __init__(self, thetas: Sequence, outs: Sequence, theta0s: Optional[Sequence] = None,
                 grad_sims: Optional[Sequence] = None, grad_thetas: Optional[Sequence] = None,
                 tensor_ids: Optional[Sequence[int]] = None, elem_offsets: Optional[Sequence[int]] = None,
                 offload: bool = False, theta0_hosts: Optional[Sequence] = None, stream=None,
                 dtypes: Optional[tuple] = None):
        torch = _torch()
        count = len(thetas)
        self.count = count
        self._refs = [thetas, outs, theta0s, grad_sims, grad_thetas, theta0_hosts]
        ids = list(tensor_ids) if tensor_ids is not None else list(range(count))
        offs = list(elem_offsets) if elem_offsets is not None else [0] * count
        if len(outs) != count or any(x is not None and len(x) != count
                                      for x in (theta0s, grad_sims, grad_thetas, theta0_hosts, tensor_ids, elem_offsets)):
            raise SmatError(SMAT_ERR_INVALID, "every per-tensor list must have one entry per tensor")
        if dtypes is None:
            t0_dt = dtype_code(theta0s[0] if theta0s is not None else outs[0]) if count else SMAT_BF16
            out_dt = dtype_code(outs[0]) if count else SMAT_BF16
            g_dt = dtype_code(grad_sims[0]) if (count and grad_sims is not None) else SMAT_BF16
        else:
            t0_dt, out_dt, g_dt = dtypes
        for i in range(count):
            n = thetas[i].numel()
            _expect(thetas[i], n, SMAT_F32, f"tensor {i}: theta")
            _expect(outs[i], n, out_dt, f"tensor {i}: out")
            if theta0s is not None:
                _expect(theta0s[i], n, t0_dt, f"tensor {i}: theta0")
            if grad_sims is not None:
                _expect(grad_sims[i], n, g_dt, f"tensor {i}: grad_sim")
            if grad_thetas is not None:
                _expect(grad_thetas[i], n, SMAT_F32, f"tensor {i}: grad_theta")
            if theta0_hosts is not None:
                _expect(theta0_hosts[i], n, t0_dt, f"tensor {i}: theta0_host")
        descs = (smat_tensor_desc * max(count, 1))()
        for i in range(count):
            d = descs[i]
            d.theta = _dev_ptr(thetas[i], "theta")
            d.out = _dev_ptr(outs[i], "out")
            d.theta0 = _dev_ptr(theta0s[i], "theta0") if theta0s is not None else None
            d.grad_sim = _dev_ptr(grad_sims[i], "grad_sim") if grad_sims is not None else None
            d.grad_theta = _dev_ptr(grad_thetas[i], "grad_theta") if grad_thetas is not None else None
            if theta0_hosts is not None:
                h = theta0_hosts[i]
                if h.is_cuda or not h.is_pinned() or not h.is_contiguous():
                    raise SmatError(SMAT_ERR_INVALID, "theta0_hosts must be contiguous pinned host tensors")
                d.theta0_host = c_void_p(h.data_ptr()) if h.numel() else None
            d.n = thetas[i].numel()
            d.tensor_id = ids[i]
            d.elem_offset = offs[i]
        self.offload = bool(offload)
        self.dtypes = (t0_dt, out_dt, g_dt)
        plan = c_void_p()
        _check(lib().smat_plan_create(descs, count, t0_dt, out_dt, g_dt, 1 if offload else 0, ctypes.byref(plan)))
        self._plan = plan
        nbytes = c_size_t()
        _check(lib().smat_plan_workspace_bytes(plan, ctypes.byref(nbytes)))
        dev = thetas[0].device if count else torch.device("cuda")
        self.workspace = torch.empty(nbytes.value, dtype=torch.uint8, device=dev)
        _check(lib().smat_plan_bind_workspace(plan, c_void_p(self.workspace.data_ptr()), nbytes.value,
                                              _stream_handle(stream)))

    def set_params(self, params, stream=None) -> None:
        """Per-tensor parameters: a sequence of dicts / smat_op_params, or an op_params_array."""
        if len(params) != self.count:
            raise SmatError(SMAT_ERR_INVALID, "one parameter record per tensor")
        if isinstance(params, np.ndarray):
            if params.dtype != OP_PARAMS_DTYPE:
                raise SmatError(SMAT_ERR_INVALID, "a parameter array must have OP_PARAMS_DTYPE records")
            arr = np.ascontiguousarray(params)
            ptr = arr.ctypes.data_as(POINTER(smat_op_params)) if self.count else None
        else:
            ptr = (smat_op_params * max(self.count, 1))(*[op_params(p) for p in params])
        _check(lib().smat_plan_set_params(self._plan, ptr, _stream_handle(stream)))

    def simulate(self, seed: int, step: int, stream=None) -> None:
        _check(lib().smat_simulate_multi(self._plan, int(seed), int(step), _stream_handle(stream)))

    def backward_accum(self, seed: int, step: int, lam: float, stream=None) -> None:
        _check(lib().smat_backward_accum_multi(self._plan, int(seed), int(step), float(lam), _stream_handle(stream)))

    def simulate_dev(self, state, stream=None) -> None:
        """smat_simulate_multi_dev: seed, step and scale read from `state` when the kernels run."""
        _check(lib().smat_simulate_multi_dev(self._plan, _state_ptr(state), _stream_handle(stream)))

    def backward_dev(self, state, lam: float, accumulate: bool = True, stream=None) -> None:
        """smat_backward_multi_dev: the backward of the step whose seed, step and scale `state` holds."""
        _check(lib().smat_backward_multi_dev(self._plan, _state_ptr(state), float(lam), 1 if accumulate else 0,
                                             _stream_handle(stream)))

    def backward(self, seed: int, step: int, lam: float, accumulate: bool = True, stream=None) -> None:
        """smat_backward_multi: accumulate into grad_theta, or overwrite it (zero where dropped)."""
        _check(lib().smat_backward_multi(self._plan, int(seed), int(step), float(lam), 1 if accumulate else 0,
                                         _stream_handle(stream)))

    def set_grads(self, grad_sims: Optional[Sequence] = None, grad_thetas: Optional[Sequence] = None,
                  stream=None) -> None:
        """Point the plan at new gradient tensors (smat_plan_set_grads); None keeps that kind as it
        is.  Holds the tensors until they are replaced."""
        arrays = []
        for ts, what, dt in ((grad_sims, "grad_sim", self.dtypes[2]), (grad_thetas, "grad_theta", SMAT_F32)):
            if ts is None:
                arrays.append(None)
                continue
            if len(ts) != self.count:
                raise SmatError(SMAT_ERR_INVALID, f"one {what} per tensor")
            for i, (g, th) in enumerate(zip(ts, self._refs[0])):
                _expect(g, th.numel(), dt, f"tensor {i}: {what}")
            arrays.append((c_void_p * max(self.count, 1))(*[_dev_ptr(g, what) for g in ts]))
        _check(lib().smat_plan_set_grads(self._plan, arrays[0], arrays[1], _stream_handle(stream)))
        if grad_sims is not None:
            self._refs[3] = list(grad_sims)
        if grad_thetas is not None:
            self._refs[4] = list(grad_thetas)

    def clear_grads(self, grad_sims: bool = True, grad_thetas: bool = True) -> None:
        """Forget the plan's gradient arrays of the chosen kinds (smat_plan_clear_grads) and drop
        the references the plan object held to them."""
        which = (1 if grad_sims else 0) | (2 if grad_thetas else 0)
        if which:
            _check(lib().smat_plan_clear_grads(self._plan, which))
        if grad_sims:
            self._refs[3] = None
        if grad_thetas:
            self._refs[4] = None

    def bind_adam_state(self, exp_avgs: Sequence, exp_avg_sqs: Sequence, stream=None) -> None:
        if len(exp_avgs) != self.count or len(exp_avg_sqs) != self.count:
            raise SmatError(SMAT_ERR_INVALID, "one optimizer state per tensor")
        for i, (a, b, th) in enumerate(zip(exp_avgs, exp_avg_sqs, self._refs[0])):
            _expect(a, th.numel(), SMAT_F32, f"tensor {i}: exp_avg")
            _expect(b, th.numel(), SMAT_F32, f"tensor {i}: exp_avg_sq")
        arr = (smat_adam_state * max(self.count, 1))(
            *[smat_adam_state(_dev_ptr(a, "exp_avg"), _dev_ptr(b, "exp_avg_sq")) for a, b in zip(exp_avgs, exp_avg_sqs)])
        self._refs.append((exp_avgs, exp_avg_sqs))
        _check(lib().smat_plan_bind_adam_state(self._plan, arr, _stream_handle(stream)))

    def adamw_fused(self, seed: int, step: int, lam: float, hp, accumulate: bool = False, grad_scale_dev=None,
                    stream=None) -> None:
        _check(lib().smat_adamw_fused_multi(self._plan, int(seed), int(step), float(lam), adamw_params(hp),
                                            1 if accumulate else 0,
                                            _scalar_ptr(grad_scale_dev, "grad_scale_dev", "float32"),
                                            _stream_handle(stream)))

    def grad_norm(self, seed: int, step: int, lam: float, accumulate: bool = False, max_norm: float = 0.0,
                  sumsq=None, clip_coef=None, stream=None) -> None:
        """smat_grad_norm_multi: the squared norm of the expert gradient into `sumsq` (one-element
        fp64 GPU tensor) and/or the clipping factor for `max_norm` into `clip_coef` (fp32)."""
        _check(lib().smat_grad_norm_multi(self._plan, int(seed), int(step), float(lam), 1 if accumulate else 0,
                                          float(max_norm), _scalar_ptr(sumsq, "sumsq", "float64"),
                                          _scalar_ptr(clip_coef, "clip_coef", "float32"), _stream_handle(stream)))

    def adamw_fused_dev(self, state, adam_state, lam: float, hp, accumulate: bool = False, grad_scale_dev=None,
                        stream=None) -> None:
        """smat_adamw_fused_multi_dev: seed, step and scale from `state`, lr and the optimizer's step
        count from `adam_state` (an AdamStepState); hp gives the other hyperparameters."""
        if isinstance(hp, dict):
            hp = dict(dict(lr=0.0, step=1), **hp)
        _check(lib().smat_adamw_fused_multi_dev(self._plan, _state_ptr(state),
                                                _state_ptr(adam_state, AdamStepState, 8, "optimizer step state"),
                                                adamw_params(hp), float(lam), 1 if accumulate else 0,
                                                _scalar_ptr(grad_scale_dev, "grad_scale_dev", "float32"),
                                                _stream_handle(stream)))

    def grad_norm_dev(self, state, lam: float, accumulate: bool = False, max_norm: float = 0.0, sumsq=None,
                      clip_coef=None, stream=None) -> None:
        """smat_grad_norm_multi_dev: grad_norm with seed, step and scale read from `state`."""
        _check(lib().smat_grad_norm_multi_dev(self._plan, _state_ptr(state), float(lam), 1 if accumulate else 0,
                                              float(max_norm), _scalar_ptr(sumsq, "sumsq", "float64"),
                                              _scalar_ptr(clip_coef, "clip_coef", "float32"), _stream_handle(stream)))

    def switch_storage(self, to: int, stream=None) -> None:
        # the stream orders only the offload prefetch; a resident plan's switch enqueues nothing
        handle = _stream_handle(stream) if (self.offload or stream is not None) else None
        _check(lib().smat_switch_storage(self._plan, int(to), handle))

    @property
    def state(self) -> int:
        st = c_int32()
        _check(lib().smat_plan_state(self._plan, ctypes.byref(st)))
        return st.value

    def active_ptrs(self):
        """(host list of active pointers, device address of the active pointer table)."""
        host = (c_void_p * max(self.count, 1))()
        dev = c_void_p()
        _check(lib().smat_plan_active_ptrs(self._plan, host, ctypes.byref(dev)))
        return [host[i] or 0 for i in range(self.count)], dev.value or 0

    def close(self) -> None:
        if getattr(self, "_plan", None):
            _check(lib().smat_plan_destroy(self._plan))
            self._plan = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


# ------------------------------------------------------------------ N-expert merge
def merge_term(t) -> smat_merge_term:
    """dict(gamma, keep=1, rescale=1, seed=0, step=0) or an smat_merge_term -> smat_merge_term."""
    if isinstance(t, smat_merge_term):
        return t
    return smat_merge_term(float(t["gamma"]), float(t.get("keep", 1.0)), int(t.get("rescale", 1)),
                           int(t.get("step", 0)), int(t.get("seed", 0)))


def smat_merge(experts: Sequence, theta0, out, terms: Sequence, tensor_id: int = 0, elem_offset: int = 0,
               stream=None) -> None:
    """out = theta0 + sum_j gamma_j m_j (experts[j] - theta0) for one flat tensor (see include/smat.h)."""
    n = out.numel()
    if theta0.numel() != n or any(x.numel() != n for x in experts):
        raise SmatError(SMAT_ERR_INVALID, "experts, theta0 and out differ in size")
    if len(terms) != len(experts) or not experts:
        raise SmatError(SMAT_ERR_INVALID, "one term per expert, at least one expert")
    dts = {dtype_code(x) for x in experts}
    if len(dts) != 1:
        raise SmatError(SMAT_ERR_DTYPE, "all experts must share one dtype")
    ptrs = (c_void_p * len(experts))(*[_dev_ptr(x, "expert") for x in experts])
    arr = (smat_merge_term * len(terms))(*[merge_term(t) for t in terms])
    _check(lib().smat_merge(ptrs, len(experts), dts.pop(), _dev_ptr(theta0, "theta0"), dtype_code(theta0),
                            _dev_ptr(out, "out"), dtype_code(out), n, arr, int(tensor_id), int(elem_offset),
                            _stream_handle(stream)))


class MergePlan:
    """A tensor list merged from N experts by one launch per call (smat_merge_plan_* calls).
    experts[j][i] is expert j's version of tensor i; holds references to every tensor."""

    def __init__(self, theta0s: Sequence, outs: Sequence, experts: Sequence[Sequence],
                 tensor_ids: Optional[Sequence[int]] = None, elem_offsets: Optional[Sequence[int]] = None,
                 stream=None):
        torch = _torch()
        count, nexp = len(theta0s), len(experts)
        if nexp == 0 or any(len(e) != count for e in experts) or len(outs) != count:
            raise SmatError(SMAT_ERR_INVALID, "experts[j] and outs must list every tensor")
        self.count, self.nexp = count, nexp
        self._refs = [theta0s, outs, experts]
        ids = list(tensor_ids) if tensor_ids is not None else list(range(count))
        offs = list(elem_offsets) if elem_offsets is not None else [0] * count
        if count:
            dts = {dtype_code(experts[j][i]) for j in range(nexp) for i in range(count)}
            if len(dts) != 1:
                raise SmatError(SMAT_ERR_DTYPE, "all experts must share one dtype")
            e_dt, t0_dt, out_dt = dts.pop(), dtype_code(theta0s[0]), dtype_code(outs[0])
        else:
            e_dt = t0_dt = out_dt = SMAT_BF16
        for i in range(count):
            n = theta0s[i].numel()
            _expect(theta0s[i], n, t0_dt, f"tensor {i}: theta0")
            _expect(outs[i], n, out_dt, f"tensor {i}: out")
            for j in range(nexp):
                _expect(experts[j][i], n, e_dt, f"tensor {i}: expert {j}")
        descs = (smat_merge_desc * max(count, 1))()
        ptrs = (c_void_p * max(count * nexp, 1))()
        for i in range(count):
            n = theta0s[i].numel()
            d = descs[i]
            d.theta0 = _dev_ptr(theta0s[i], "theta0")
            d.out = _dev_ptr(outs[i], "out")
            d.n = n
            d.tensor_id = ids[i]
            d.elem_offset = offs[i]
            for j in range(nexp):
                ptrs[i * nexp + j] = _dev_ptr(experts[j][i], "expert")
        plan = c_void_p()
        _check(lib().smat_merge_plan_create(descs, count, ptrs, nexp, e_dt, t0_dt, out_dt, ctypes.byref(plan)))
        self._plan = plan
        nbytes = c_size_t()
        _check(lib().smat_merge_plan_workspace_bytes(plan, ctypes.byref(nbytes)))
        dev = theta0s[0].device if count else torch.device("cuda")
        self.workspace = torch.empty(nbytes.value, dtype=torch.uint8, device=dev)
        _check(lib().smat_merge_plan_bind_workspace(plan, c_void_p(self.workspace.data_ptr()), nbytes.value,
                                                    _stream_handle(stream)))

    def merge(self, terms: Sequence, stream=None) -> None:
        """terms: one per expert (applied to every tensor), or a list per tensor of one per expert."""
        if len(terms) and isinstance(terms[0], (list, tuple)):
            if len(terms) != self.count or any(len(r) != self.nexp for r in terms):
                raise SmatError(SMAT_ERR_INVALID, "one row of terms per tensor, one term per expert")
            flat = [merge_term(t) for row in terms for t in row]
        else:
            if len(terms) != self.nexp:
                raise SmatError(SMAT_ERR_INVALID, "one term per expert")
            flat = [merge_term(t) for _ in range(self.count) for t in terms]
        arr = (smat_merge_term * max(len(flat), 1))(*flat)
        _check(lib().smat_merge_multi(self._plan, arr, _stream_handle(stream)))

    def close(self) -> None:
        if getattr(self, "_plan", None):
            _check(lib().smat_merge_plan_destroy(self._plan))
            self._plan = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def smat_stream_copy(src, dst, stream=None) -> None:
    """Plain streaming copy src -> dst (same byte size, GPU tensors; the HBM reference)."""
    nb = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nb:
        raise SmatError(SMAT_ERR_INVALID, "src and dst differ in size")
    _check(lib().smat_stream_copy(_dev_ptr(src, "src"), _dev_ptr(dst, "dst"), nb, _stream_handle(stream)))
