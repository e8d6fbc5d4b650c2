"""SMAT inside a PyTorch training loop (Sec. 4.3): periodic simulated steps with storage switching.

Each cycle of t steps has t - 1 ordinary steps and one simulated step (step mod t == t - 1).
Each step computes one loss with one forward and one backward pass.  On a simulated step:

1. `begin(step)` draws one scale alpha ~ U[alpha_min, 1] for all tensors (Sec. 4.1, Scale) from
   (seed, step) (smat_scale_draw, the generator's scale stream),
   writes theta~ = theta0 + alpha m (.) (theta - theta0) + eps into one reusable buffer per
   parameter (smat_simulate_multi), and rebinds each parameter's `.data` to its buffer.  The
   model's forward and backward then run on theta~; autograd's gradient tensors at theta~ are
   handed to the library as they are (smat_plan_set_grads), with no copy.
2. `end(optimizer)` turns that gradient into the expert gradient lambda alpha m (.) g~
   (Eq. smat-gradient), with the mask regenerated (smat_backward_accum_multi).  It then rebinds
   `.data` to the expert storage, so that the optimizer, weight decay included, only sees the fp32
   expert weights (App. "Training and Scheduling Details", "Implementation details").  With
   `fused=True` it applies the torch Adam/AdamW update instead, straight from g~, on that optimizer's
   own moment tensors (smat_adamw_fused_multi).  No gradient tensor is written, and the caller
   skips `optimizer.step()` for that step.

A gradient already in p.grad when `begin` runs (the expert loss's backward in the same step) is
kept, and the simulated-loss gradient is added to it: the objective (1 - lam) L(theta) +
lam L(theta~) of Eq. smat-objective with both losses every step, when the caller scales the expert
loss by 1 - lam.  Periodic scheduling instead calls `begin` after zero_grad().

Ordinary steps touch nothing.  In offload mode theta0 stays in pinned host memory.  The restore
at the end of each simulated step starts the copy of theta0 into the buffers on the library's copy
stream, and that copy runs during the following ordinary steps.  The arithmetic runs in libsmat.
This module only rebinds tensors and sequences library calls.
"""
from __future__ import annotations

from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import _lib
from ._lib import (SMAT_ERR_INVALID, SMAT_ERR_STATE, SMAT_EXPERT, SMAT_NOISE_UNIFORM, SMAT_SIMULATED, Plan,
                   SmatError)

DEFAULT_HEAD_NAMES = ("lm_head", "head", "classifier", "output")


def is_simulated_step(step: int, period: int) -> bool:
    """t - 1 ordinary steps, then one simulated step: step mod t == t - 1 (0-based steps), so the
    ordinary steps of a cycle come first (Sec. 4.3, Periodic scheduling)."""
    if period < 1 or step < 0:
        raise SmatError(SMAT_ERR_INVALID, "period must be >= 1 and step >= 0")
    return step % period == period - 1


def mask_set(model: torch.nn.Module, head_names: Iterable[str] = DEFAULT_HEAD_NAMES
             ) -> List[Tuple[str, torch.nn.Parameter, bool]]:
    """(name, parameter, in S) for every trainable parameter, shared ones once.

    S, the set the Mask applies to, holds the weights of the attention and MLP linear layers
    (Sec. 4.1, Mask): the `weight` of every nn.Linear whose module name does not end in one of
    `head_names`, and which is not also the weight of an nn.Embedding (tied output layers).
    Biases, norms, embeddings and output heads are outside S (no drop, keep = 1)."""
    heads = tuple(head_names)
    embed = {id(m.weight) for m in model.modules() if isinstance(m, torch.nn.Embedding)}
    linear = set()
    for mname, m in model.named_modules():
        if isinstance(m, torch.nn.Linear) and mname.split(".")[-1] not in heads and id(m.weight) not in embed:
            linear.add(id(m.weight))
    return [(n, p, id(p) in linear) for n, p in model.named_parameters() if p.requires_grad]


def adam_hparams(optimizer: torch.optim.Optimizer, params: Sequence[torch.nn.Parameter]) -> dict:
    """lr, beta1, beta2, eps, weight_decay and the next 1-based step k shared by `params` in a torch
    Adam or AdamW optimizer, for the fused update.  Raises SmatError(SMAT_ERR_INVALID) when the
    update is not the decoupled-weight-decay Adam the kernel computes (amsgrad, maximize, Adam's
    L2-coupled weight decay), when the parameters' groups disagree, or when their step counts do."""
    if not isinstance(optimizer, (torch.optim.Adam, torch.optim.AdamW)):
        raise SmatError(SMAT_ERR_INVALID, "the fused update needs a torch.optim.Adam or AdamW optimizer")
    where = {}
    for gi, group in enumerate(optimizer.param_groups):
        for p in group["params"]:
            where[id(p)] = gi
    keys = set()
    for p in params:
        if id(p) not in where:
            raise SmatError(SMAT_ERR_INVALID, "a parameter is not in the optimizer")
        keys.add(where[id(p)])
    hps = []
    for gi in sorted(keys):
        g = optimizer.param_groups[gi]
        if g.get("amsgrad", False) or g.get("maximize", False):
            raise SmatError(SMAT_ERR_INVALID, "amsgrad and maximize are not supported by the fused update")
        wd = float(g["weight_decay"])
        coupled = isinstance(optimizer, torch.optim.Adam) and not isinstance(optimizer, torch.optim.AdamW) \
            and not g.get("decoupled_weight_decay", False)
        if coupled and wd != 0.0:
            raise SmatError(SMAT_ERR_INVALID, "Adam's L2 weight decay is not supported by the fused update")
        b1, b2 = g["betas"]
        hps.append((float(g["lr"]), float(b1), float(b2), float(g["eps"]), wd))
    if len(set(hps)) > 1:
        raise SmatError(SMAT_ERR_INVALID, "parameters of the fused update must share lr, betas, eps and weight decay")
    steps = set()
    for p in params:
        st = optimizer.state.get(p)
        steps.add(int(float(st["step"])) if st and "step" in st else 0)
    if len(steps) > 1:
        raise SmatError(SMAT_ERR_INVALID, "parameters of the fused update must share the optimizer step count")
    lr, b1, b2, eps, wd = hps[0] if hps else (0.0, 0.9, 0.999, 1e-8, 0.0)
    return dict(lr=lr, beta1=b1, beta2=b2, eps=eps, weight_decay=wd, step=steps.pop() + 1 if steps else 1)


class SimulatedMergeTraining:
    """Periodic simulated-merge steps over a list of trainable fp32 parameters.

    params        trainable parameters (fp32, contiguous, on one GPU): the expert storage
    theta0        frozen base weights, one per parameter, same shapes (copied to `buffer_dtype`)
    keep          per-parameter keep probability 1 - p; 1 outside the mask set S
    alpha_min     lower bound of the scale alpha ~ U[alpha_min, 1] (one draw per simulated step)
    sigma         Perturb RMS, one value or one per parameter
    period        t: one simulated step per t steps (Sec. 4.3, Periodic scheduling)
    lam           weight of the simulated-loss gradient (1: the step computes only that loss)
    noise_kind    SMAT_NOISE_UNIFORM (the method's default), _GAUSSIAN or _LAPLACE
    rescale       multiply kept coordinates by 1/keep (Eq. smat-mask)
    buffer_dtype  dtype of theta~ and of its gradient (bf16 halves the buffer; fp32 for fp32 models)
    offload       keep theta0 in pinned host memory and prefetch it into the buffers at each restore
    """

    def __init__(self, params: Sequence[torch.nn.Parameter], theta0: Sequence[torch.Tensor], keep: Sequence[float],
                 alpha_min: float, sigma, period: int = 4, lam: float = 1.0, seed: int = 0,
                 noise_kind: int = SMAT_NOISE_UNIFORM, rescale: bool = True,
                 buffer_dtype: torch.dtype = torch.bfloat16, offload: bool = False):
        self.plan = None
        self.params = list(params)
        n = len(self.params)
        if n == 0:
            raise SmatError(SMAT_ERR_INVALID, "no parameters")
        if period < 1 or not (0.0 <= alpha_min <= 1.0):
            raise SmatError(SMAT_ERR_INVALID, "period must be >= 1 and alpha_min in [0, 1]")
        if len(theta0) != n or len(keep) != n:
            raise SmatError(SMAT_ERR_INVALID, "one theta0 and one keep per parameter")
        dev = self.params[0].device
        for p, t0 in zip(self.params, theta0):
            if p.dtype != torch.float32 or p.device != dev or not p.data.is_contiguous() or not p.is_cuda:
                raise SmatError(SMAT_ERR_INVALID, "parameters must be contiguous fp32 tensors on one GPU")
            if tuple(t0.shape) != tuple(p.shape):
                raise SmatError(SMAT_ERR_INVALID, "theta0 must match its parameter's shape")
        if buffer_dtype not in (torch.float32, torch.bfloat16):
            raise SmatError(_lib.SMAT_ERR_DTYPE, "buffer_dtype must be float32 or bfloat16")
        self.master = [p.data for p in self.params]
        self.keep = [float(k) for k in keep]
        self.sigma = [float(sigma)] * n if np.ndim(sigma) == 0 else [float(x) for x in sigma]
        if len(self.sigma) != n:
            raise SmatError(SMAT_ERR_INVALID, "one sigma per parameter")
        self.alpha_min, self.period, self.lam, self.seed = float(alpha_min), int(period), float(lam), int(seed)
        self.noise_kind, self.rescale, self.offload = int(noise_kind), 1 if rescale else 0, bool(offload)
        # the only resident state: one buffer per parameter (plus theta0 unless offloaded).  Gradient
        # arrays are the step's own tensors, handed to the plan when they exist.
        self.buffers = [torch.empty(p.shape, dtype=buffer_dtype, device=dev) for p in self.params]
        dt = _lib.dtype_code(self.buffers[0])
        if self.offload:
            self.theta0_host = [t.detach().to("cpu", dtype=buffer_dtype).contiguous().pin_memory() for t in theta0]
            self.plan = Plan(self.master, self.buffers, None, offload=True, theta0_hosts=self.theta0_host,
                             dtypes=(dt, dt, dt))
        else:
            self.theta0 = [t.detach().to(device=dev, dtype=buffer_dtype).contiguous() for t in theta0]
            self.plan = Plan(self.master, self.buffers, self.theta0, dtypes=(dt, dt, dt))
        self.alpha: Optional[float] = None      # the scale of the current (or last) simulated step
        self._step: Optional[int] = None        # set between begin() and end()
        self._adam_key = None
        self._clip = None                       # GPU scalars (sumsq, clipping factor) of the fused update
        self._grads = None                      # gradients at theta~ the plan points at
        self._expert_grads = None               # the expert loss's gradients of the open step, if any
        self.names = [f"param{i}" for i in range(n)]

    @classmethod
    def from_module(cls, model: torch.nn.Module, keep: float = 0.5, alpha_min: float = 0.2, sigma: float = 2e-3,
                    theta0: Optional[dict] = None, head_names: Iterable[str] = DEFAULT_HEAD_NAMES, **kw):
        """Wrap every trainable parameter of `model`: keep `keep` inside S (see mask_set), 1 outside.
        theta0 defaults to the current weights (wrap right after loading the base model); otherwise a
        dict name -> tensor.  Defaults are the method's LLM settings (p = 0.5, alpha_min = 0.2,
        sigma = 2e-3, t = 4)."""
        entries = mask_set(model, head_names)
        names = [n for n, _, _ in entries]
        params = [p for _, p, _ in entries]
        t0 = [p.detach() for p in params] if theta0 is None else [theta0[n] for n in names]
        wrapper = cls(params, t0, [keep if s else 1.0 for _, _, s in entries], alpha_min, sigma, **kw)
        wrapper.names = names
        return wrapper

    # ------------------------------------------------------------------ schedule
    def is_simulated(self, step: int) -> bool:
        return is_simulated_step(step, self.period)

    @property
    def active(self) -> bool:
        return self._step is not None

    # ------------------------------------------------------------------ simulated step
    def begin(self, step: int) -> bool:
        """Call before the forward pass of the simulated loss: after zero_grad() (periodic
        scheduling), or after the expert loss's backward to add both gradients.  On a simulated step,
        point the parameters at theta~; returns whether the step is simulated."""
        if self._step is not None:
            raise SmatError(SMAT_ERR_STATE, "begin() while a simulated step is open")
        if not self.is_simulated(step):
            return False
        # alpha is a function of (seed, step), like the masks and the noise: a resumed run draws the same
        self.alpha = _lib.scale_draw(self.seed, step, self.alpha_min)
        self.plan.set_params(_lib.op_params_array(len(self.params), self.alpha, self.keep, self.sigma, self.rescale,
                                                  self.noise_kind))
        self.plan.simulate(self.seed, step)
        self.plan.switch_storage(SMAT_SIMULATED)
        self._grads = None      # last step's gradients, no longer read by any queued kernel
        self._expert_grads = None
        if any(p.grad is not None for p in self.params):   # the expert loss's gradient of this step
            self._expert_grads = [None if p.grad is None else
                                  p.grad.to(dtype=torch.float32, memory_format=torch.contiguous_format)
                                  for p in self.params]
        for p, b in zip(self.params, self.buffers):
            p.data = b
            p.grad = None       # autograd creates the gradient at theta~ and keeps it as p.grad
        self._step = int(step)
        return True

    def _grads_at_theta_tilde(self) -> List[torch.Tensor]:
        """The gradients at theta~ that autograd left in p.grad (zeros for unused parameters)."""
        grads = []
        for p, b in zip(self.params, self.buffers):
            g = p.grad
            if g is None:                            # the parameter took no part in the loss
                g = torch.zeros_like(b)
            elif not g.is_contiguous() or g.dtype != b.dtype:
                g = g.to(dtype=b.dtype, memory_format=torch.contiguous_format)
            grads.append(g)
        return grads

    def _restore(self) -> None:
        self.plan.switch_storage(SMAT_EXPERT)
        for p, m in zip(self.params, self.master):
            p.data = m
            p.grad = None
        self._step = None

    def end(self, optimizer: Optional[torch.optim.Optimizer] = None, fused: bool = False,
            grad_scale: float = 1.0, max_norm: Optional[float] = None) -> Optional[torch.Tensor]:
        """Call after the backward pass of a simulated step.  Without `fused`, leaves
        param.grad = lam * alpha * m (.) g~ on the expert storage for the caller's optimizer.step()
        (and its own clipping).  With `fused`, applies the update of `optimizer` (torch Adam/AdamW)
        directly; its hyperparameters and step count come from that optimizer, `grad_scale`
        multiplies the gradient, and the caller must not call optimizer.step().  With `max_norm`
        the fused update first clips the expert gradient to that L2 norm as
        torch.nn.utils.clip_grad_norm_ would (smat_grad_norm_multi, factor kept on the GPU); the
        gradient's total norm is then returned as a GPU scalar."""
        if self._step is None:
            raise SmatError(SMAT_ERR_STATE, "end() without an open simulated step")
        if max_norm is not None and not fused:
            raise SmatError(SMAT_ERR_INVALID, "max_norm applies to the fused update; clip param.grad otherwise")
        step = self._step
        grads = self._grads_at_theta_tilde()
        if fused:
            if optimizer is None:
                raise SmatError(SMAT_ERR_INVALID, "the fused update needs the optimizer that owns the moments")
            hp = adam_hparams(optimizer, self.params)   # validate before touching any state
            wrapped = {id(p) for p in self.params}
            if any(id(q) not in wrapped and q.grad is not None for g in optimizer.param_groups for q in g["params"]):
                raise SmatError(SMAT_ERR_INVALID, "the optimizer holds parameters outside the wrapper that have "
                                                  "gradients; the fused update would skip them")
            self._restore()
            acc = self._accumulator(zeros=False)
            self.plan.set_grads(grads, acc)
            self._grads = grads     # kept alive until the kernels that read them have been queued
            norm = self._fused_adam(optimizer, dict(hp, grad_scale=float(grad_scale)), step, max_norm,
                                    accumulate=acc is not None)
            self.plan.clear_grads()  # this step's gradient tensors may be freed from here on
            return norm
        # the expert gradient is written into fresh fp32 tensors, as an ordinary step's gradients
        # are, or added to the expert loss's gradient of this step
        acc = self._accumulator(zeros=False)
        expert = acc if acc is not None else [torch.empty_like(m) for m in self.master]
        self.plan.set_grads(grads, expert)
        self._grads = grads
        self.plan.backward(self.seed, step, self.lam, accumulate=acc is not None)
        self.plan.clear_grads()      # the caller frees these tensors (zero_grad) after its optimizer step
        self._restore()
        for p, g in zip(self.params, expert):
            p.grad = g
        return None

    def _accumulator(self, zeros: bool) -> Optional[List[torch.Tensor]]:
        """fp32 gradients the simulated-loss gradient is added to: the expert loss's gradients kept
        by begin() (zeros where a parameter had none); without them, fresh zeros when `zeros`, else
        None."""
        if self._expert_grads is None:
            return [torch.zeros_like(m) for m in self.master] if zeros else None
        acc = [torch.zeros_like(m) if g is None else g for g, m in zip(self._expert_grads, self.master)]
        self._expert_grads = None
        return acc

    def abort(self) -> None:
        """Leave an open simulated step without any update (e.g. after an exception or a skipped
        step): the expert storage is restored, the gradients at theta~ are dropped and the expert
        loss's gradients kept by begin() are put back.  No-op when no step is open."""
        if self._step is not None:
            self._restore()
            if self._expert_grads is not None:
                for p, g in zip(self.params, self._expert_grads):
                    p.grad = g
                self._expert_grads = None

    def _fused_adam(self, optimizer, hp: dict, step: int, max_norm: Optional[float],
                    accumulate: bool = False) -> Optional[torch.Tensor]:
        exp_avg, exp_avg_sq, counts = [], [], []
        for p in self.params:
            st = optimizer.state[p]
            if "exp_avg" not in st:   # first update: the state torch's Adam would create
                group = next(g for g in optimizer.param_groups if any(q is p for q in g["params"]))
                on_dev = group.get("fused") or group.get("capturable")
                st["step"] = (torch.zeros((), dtype=torch.float32, device=p.device) if on_dev
                              else torch.tensor(0.0, dtype=torch.float32))
                st["exp_avg"] = torch.zeros_like(p, memory_format=torch.preserve_format)
                st["exp_avg_sq"] = torch.zeros_like(p, memory_format=torch.preserve_format)
            exp_avg.append(st["exp_avg"])
            exp_avg_sq.append(st["exp_avg_sq"])
            counts.append(st["step"])
        key = tuple(t.data_ptr() for t in exp_avg + exp_avg_sq)
        if key != self._adam_key:
            self.plan.bind_adam_state(exp_avg, exp_avg_sq)
            self._adam_key = key
        coef = norm = None
        if max_norm is not None:
            if self._clip is None:
                dev = self.master[0].device
                self._clip = (torch.zeros(1, dtype=torch.float64, device=dev), torch.ones(1, dtype=torch.float32, device=dev))
            sumsq, coef = self._clip
            self.plan.grad_norm(self.seed, step, self.lam, accumulate, float(max_norm), sumsq, coef)
            norm = sumsq.sqrt()
        self.plan.adamw_fused(self.seed, step, self.lam, hp, accumulate=accumulate, grad_scale_dev=coef)
        for c in counts:        # the optimizer's own step counts (CPU or GPU scalars)
            c.add_(1)
        return norm

    def close(self) -> None:
        if self.plan is not None:
            self.abort()
            self.plan.close()
            self.plan = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
