"""Seeded synthetic parameter lists shaped like the backbones SMAT trains.

This module only builds inputs: tensor shapes, seeded values and per-tensor
settings (scale, keep probability, noise RMS).  It holds none of the method's
arithmetic, so both the HIP path and the CPU oracle can consume what it makes.

Workloads (all parameters synthetic, no checkpoints):

* ``c1``   one flat fp32 tensor of 1,048,576 elements (theta0 = theta + N(0, 0.01^2)).
* ``c2``   200 tensors, 123,730,176 params, a 12-layer d=768 GPT-2-style stack.
* ``c3``   254 tensors, 1,543,656,960 params, a 28-layer d=1536 GQA decoder
           (SwiGLU 8960, vocab 151936), simulated every 4th step.
* ``c4``   290 tensors, 7,504,924,672 params, a 32-layer d=4096 GQA decoder
           (SwiGLU 14336, vocab 128256).
* ``c5``   ~1,825 tensors, ~7.83e9 params: a ViT-L/14-shaped tower, a 2-layer
           projector and the c4 decoder, plus 1,236 seeded small vectors.
* ``mini`` a small ragged list (several kernel tiles, odd sizes and tails) that
           the CPU oracle checks element by element in seconds.

Paper context: the mask set S is the linear weights of attention and MLP
blocks; biases, norms and embeddings are not masked (Sec. 4.1, "Mask").
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

# kinds of parameter tensors
LINEAR = "linear"      # attention / MLP / projector linear weights: the mask set S
EMBED = "embed"        # token embedding (tied head)
NORM_W = "norm_w"      # norm gains (init around 1)
BIAS = "bias"          # biases and norm shifts
CONV = "conv"          # patch embedding
POS = "pos"            # position embedding
CLS = "cls"            # class token
EXTRA = "extra"        # padding vectors that bring a list to its stated count
FLAT = "flat"          # c1's single flat tensor

MATRIX_KINDS = (LINEAR, EMBED, CONV, POS, CLS)


@dataclass(frozen=True)
class TensorSpec:
    name: str
    shape: tuple
    kind: str

    @property
    def numel(self) -> int:
        return int(np.prod(self.shape, dtype=np.int64))


@dataclass
class Config:
    name: str
    index: int
    specs: List[TensorSpec]
    theta0_dtype: str          # "bf16" or "f32"
    grad_dtype: str            # dtype of the upstream gradient g~
    out_dtype: str             # dtype of the simulated weights
    delta_std: float           # std of theta - theta0
    sigma_mult: Optional[float]  # sigma = sigma_mult * std(theta - theta0); None => fixed sigma
    sigma_fixed: float
    s_range: tuple             # scale s ~ U[lo, hi]; lo == hi => fixed
    keep_rule: str             # "fixed", "uniform", "split"
    keep_value: float
    keep_range: tuple
    lam: float
    period: int                # simulate every `period`-th step (1 => every step)
    description: str = ""

    @property
    def data_seed(self) -> int:
        return self.index

    @property
    def smat_seed(self) -> int:
        return 0x5EED0000 + self.index

    @property
    def numel(self) -> int:
        return sum(s.numel for s in self.specs)

    @property
    def count(self) -> int:
        return len(self.specs)


# ----------------------------------------------------------------- shapes

def _gpt2_small_specs() -> List[TensorSpec]:
    d, ff, vocab = 768, 3072, 50304
    out: List[TensorSpec] = []
    for l in range(12):
        p = f"h{l}."
        out += [
            TensorSpec(p + "attn.qkv.w", (d, 3 * d), LINEAR),
            TensorSpec(p + "attn.qkv.b", (3 * d,), BIAS),
            TensorSpec(p + "attn.proj.w", (d, d), LINEAR),
            TensorSpec(p + "attn.proj.b", (d,), BIAS),
            TensorSpec(p + "mlp.fc.w", (d, ff), LINEAR),
            TensorSpec(p + "mlp.fc.b", (ff,), BIAS),
            TensorSpec(p + "mlp.proj.w", (ff, d), LINEAR),
            TensorSpec(p + "mlp.proj.b", (d,), BIAS),
            TensorSpec(p + "ln1.w", (d,), NORM_W),
            TensorSpec(p + "ln1.b", (d,), BIAS),
            TensorSpec(p + "ln2.w", (d,), NORM_W),
            TensorSpec(p + "ln2.b", (d,), BIAS),
        ]
    out.append(TensorSpec("wte", (vocab, d), EMBED))
    out.append(TensorSpec("ln_f.w", (d,), NORM_W))
    out.append(TensorSpec("ln_f.b", (d,), BIAS))
    while len(out) < 200:
        out.append(TensorSpec(f"extra{len(out)}", (d,), EXTRA))
    return out


def _decoder_specs(layers: int, d: int, kv_dim: int, ff: int, vocab: int, prefix: str = "") -> List[TensorSpec]:
    out: List[TensorSpec] = []
    for l in range(layers):
        p = f"{prefix}layers.{l}."
        out += [
            TensorSpec(p + "attn.q.w", (d, d), LINEAR),
            TensorSpec(p + "attn.k.w", (kv_dim, d), LINEAR),
            TensorSpec(p + "attn.v.w", (kv_dim, d), LINEAR),
            TensorSpec(p + "attn.o.w", (d, d), LINEAR),
            TensorSpec(p + "mlp.gate.w", (ff, d), LINEAR),
            TensorSpec(p + "mlp.up.w", (ff, d), LINEAR),
            TensorSpec(p + "mlp.down.w", (d, ff), LINEAR),
            TensorSpec(p + "input_norm.w", (d,), NORM_W),
            TensorSpec(p + "post_attn_norm.w", (d,), NORM_W),
        ]
    out.append(TensorSpec(prefix + "embed_tokens", (vocab, d), EMBED))
    out.append(TensorSpec(prefix + "norm.w", (d,), NORM_W))
    return out


def _vit_l14_specs() -> List[TensorSpec]:
    d, ff = 1024, 4096
    out = [
        TensorSpec("vit.conv1.w", (d, 3, 14, 14), CONV),
        TensorSpec("vit.cls", (d,), CLS),
        TensorSpec("vit.pos", (257, d), POS),
        TensorSpec("vit.ln_pre.w", (d,), NORM_W),
        TensorSpec("vit.ln_pre.b", (d,), BIAS),
    ]
    for l in range(24):
        p = f"vit.blocks.{l}."
        out += [
            TensorSpec(p + "attn.qkv.w", (3 * d, d), LINEAR),
            TensorSpec(p + "attn.qkv.b", (3 * d,), BIAS),
            TensorSpec(p + "attn.out.w", (d, d), LINEAR),
            TensorSpec(p + "attn.out.b", (d,), BIAS),
            TensorSpec(p + "mlp.fc1.w", (ff, d), LINEAR),
            TensorSpec(p + "mlp.fc1.b", (ff,), BIAS),
            TensorSpec(p + "mlp.fc2.w", (d, ff), LINEAR),
            TensorSpec(p + "mlp.fc2.b", (d,), BIAS),
            TensorSpec(p + "ln1.w", (d,), NORM_W),
            TensorSpec(p + "ln1.b", (d,), BIAS),
            TensorSpec(p + "ln2.w", (d,), NORM_W),
            TensorSpec(p + "ln2.b", (d,), BIAS),
        ]
    out.append(TensorSpec("vit.ln_post.w", (d,), NORM_W))
    out.append(TensorSpec("vit.ln_post.b", (d,), BIAS))
    return out


def _vlm_specs() -> List[TensorSpec]:
    out = _vit_l14_specs()
    out += [
        TensorSpec("proj.fc1.w", (4096, 1024), LINEAR),
        TensorSpec("proj.fc1.b", (4096,), BIAS),
        TensorSpec("proj.fc2.w", (4096, 4096), LINEAR),
        TensorSpec("proj.fc2.b", (4096,), BIAS),
    ]
    out += _decoder_specs(32, 4096, 1024, 14336, 128256, prefix="lm.")
    # seeded small vectors (log-uniform sizes in [32, 8191]) that stress load balance
    rng = np.random.default_rng(0xC5)
    sizes = np.exp(rng.uniform(math.log(32), math.log(8192), size=1236)).astype(np.int64)
    sizes = np.clip(sizes, 32, 8191)
    extras = [TensorSpec(f"small.{i}", (int(n),), EXTRA) for i, n in enumerate(sizes)]
    # interleave the small vectors through the list so they are not all in one tail
    merged: List[TensorSpec] = []
    ei = 0
    for i, s in enumerate(out):
        merged.append(s)
        while ei < len(extras) and ei * len(out) < (i + 1) * len(extras):
            merged.append(extras[ei])
            ei += 1
    return merged


def _mini_specs() -> List[TensorSpec]:
    return [
        TensorSpec("w0", (3, 1000), LINEAR),
        TensorSpec("b0", (7,), BIAS),
        TensorSpec("w1", (257, 129), LINEAR),
        TensorSpec("n0", (4096,), NORM_W),
        TensorSpec("e0", (1000, 64), EMBED),
        TensorSpec("w2", (2048, 257), LINEAR),
        TensorSpec("v", (1,), BIAS),
        TensorSpec("w3", (5, 65537), LINEAR),
        TensorSpec("b1", (31,), BIAS),
        TensorSpec("w4", (64, 4096), LINEAR),
    ]


# ----------------------------------------------------------------- configs

def config(name: str) -> Config:
    if name == "c1":
        return Config("c1", 0, [TensorSpec("flat", (1048576,), FLAT)], "f32", "f32", "bf16",
                      delta_std=0.01, sigma_mult=None, sigma_fixed=1e-3, s_range=(0.7, 0.7),
                      keep_rule="fixed", keep_value=0.5, keep_range=(0.5, 0.5), lam=1.0, period=1,
                      description="flat fp32 tensor of 1,048,576 elements, s=0.7, keep=0.5, sigma=1e-3")
    if name == "c2":
        return Config("c2", 1, _gpt2_small_specs(), "bf16", "bf16", "bf16",
                      delta_std=1e-3, sigma_mult=0.5, sigma_fixed=0.0, s_range=(0.3, 1.0),
                      keep_rule="uniform", keep_value=0.0, keep_range=(0.1, 0.9), lam=1.0, period=1,
                      description="12-layer d=768 stack, 200 tensors, 123.7M params")
    if name == "c3":
        return Config("c3", 2, _decoder_specs(28, 1536, 256, 8960, 151936), "bf16", "bf16", "bf16",
                      delta_std=1e-3, sigma_mult=0.5, sigma_fixed=0.0, s_range=(0.3, 1.0),
                      keep_rule="fixed", keep_value=0.1, keep_range=(0.1, 0.1), lam=1.0, period=4,
                      description="28-layer d=1536 GQA decoder, 1.54B params, simulate every 4th step")
    if name == "c4":
        return Config("c4", 3, _decoder_specs(32, 4096, 1024, 14336, 128256), "bf16", "bf16", "bf16",
                      delta_std=2e-4, sigma_mult=0.3, sigma_fixed=0.0, s_range=(0.2, 1.0),
                      keep_rule="fixed", keep_value=0.2, keep_range=(0.2, 0.2), lam=0.5, period=1,
                      description="32-layer d=4096 GQA decoder, 290 tensors, 7.50B params")
    if name == "c5":
        return Config("c5", 4, _vlm_specs(), "bf16", "bf16", "bf16",
                      delta_std=2e-4, sigma_mult=0.3, sigma_fixed=0.0, s_range=(0.1, 1.0),
                      keep_rule="split", keep_value=0.2, keep_range=(0.2, 0.2), lam=0.5, period=1,
                      description="ViT-L/14 tower + projector + 7B decoder, ~1,825 tensors, 7.83B params")
    if name == "mini":
        return Config("mini", 5, _mini_specs(), "bf16", "bf16", "bf16",
                      delta_std=1e-3, sigma_mult=0.5, sigma_fixed=0.0, s_range=(0.3, 1.0),
                      keep_rule="uniform", keep_value=0.0, keep_range=(0.1, 0.9), lam=0.75, period=1,
                      description="small ragged list for element-wise parity")
    raise KeyError(name)


ALL = ("c1", "c2", "c3", "c4", "c5")


# ----------------------------------------------------------------- settings

@dataclass
class TensorSettings:
    """Per-tensor settings that stay fixed across steps."""
    keep: float        # keep probability (1 => tensor outside the mask set)
    sigma: float       # noise RMS, float32-representable
    scale_fixed: Optional[float]  # None => s drawn per step from cfg.s_range
    rescale: int = 1
    noise_kind: int = 0  # 0 = Gaussian


def static_settings(cfg: Config, sigmas: Sequence[float]) -> List[TensorSettings]:
    """keep / sigma per tensor.  `sigmas` are the data-derived noise RMS values."""
    rng = np.random.default_rng([cfg.index, 0xC0FFEE])
    out: List[TensorSettings] = []
    for i, spec in enumerate(cfg.specs):
        sig = float(np.float32(sigmas[i]))
        if cfg.keep_rule == "split":
            if i % 2 == 0:   # mask only: no scale, no noise
                out.append(TensorSettings(keep=float(np.float32(cfg.keep_value)), sigma=0.0, scale_fixed=1.0))
            else:            # scale + noise only
                out.append(TensorSettings(keep=1.0, sigma=sig, scale_fixed=None))
            continue
        masked = spec.kind in (LINEAR, FLAT)
        if not masked:
            keep = 1.0
        elif cfg.keep_rule == "uniform":
            keep = float(np.float32(rng.uniform(*cfg.keep_range)))
        else:
            keep = float(np.float32(cfg.keep_value))
        fixed = cfg.s_range[0] if cfg.s_range[0] == cfg.s_range[1] else None
        out.append(TensorSettings(keep=keep, sigma=sig, scale_fixed=fixed))
    return out


def step_scales(cfg: Config, step: int) -> np.ndarray:
    """Per-tensor scale s for one step, float32 values, seeded by (config, step)."""
    rng = np.random.default_rng([cfg.index, 0x5CA1E, int(step)])
    lo, hi = cfg.s_range
    if lo == hi:
        return np.full(cfg.count, lo, dtype=np.float32)
    return rng.uniform(lo, hi, size=cfg.count).astype(np.float32)


def step_params(cfg: Config, settings: Sequence[TensorSettings], step: int) -> List[dict]:
    """Per-tensor operation parameters for `step` as plain dicts."""
    scales = step_scales(cfg, step)
    out = []
    for i, st in enumerate(settings):
        s = st.scale_fixed if st.scale_fixed is not None else float(scales[i])
        out.append(dict(s=float(np.float32(s)), keep=st.keep, sigma=st.sigma,
                        rescale=st.rescale, noise_kind=st.noise_kind))
    return out


# ----------------------------------------------------------------- tensors

@dataclass
class Inputs:
    cfg: Config
    theta: list = field(default_factory=list)        # fp32 master weights
    theta0: list = field(default_factory=list)       # frozen base (bf16 or fp32)
    grad_sim: list = field(default_factory=list)     # upstream gradient g~ at the simulated weights
    grad_theta: list = field(default_factory=list)   # fp32 gradient accumulator
    sigmas: list = field(default_factory=list)       # float32-valued noise RMS per tensor
    settings: list = field(default_factory=list)


def _init_std(kind: str) -> tuple:
    """(mean, std) of theta0 for a tensor kind."""
    if kind == NORM_W:
        return 1.0, 0.05
    return 0.0, 0.02


def make_inputs(cfg: Config, device="cpu", with_grads: bool = True) -> Inputs:
    """Seeded tensors for `cfg` on `device` (torch).  Same seed => same values per device type."""
    import torch

    dt = {"bf16": torch.bfloat16, "f32": torch.float32}
    gen = torch.Generator(device=device)
    gen.manual_seed(cfg.data_seed)
    inp = Inputs(cfg)
    for i in range(cfg.count):
        spec = cfg.specs[i]
        shape = spec.shape
        if cfg.name == "c1":
            theta = torch.randn(shape, generator=gen, device=device, dtype=torch.float32) * 0.02
            theta0 = (theta + torch.randn(shape, generator=gen, device=device, dtype=torch.float32) * cfg.delta_std)
            theta0 = theta0.to(dt[cfg.theta0_dtype])
        else:
            mean, std = _init_std(spec.kind)
            base = torch.randn(shape, generator=gen, device=device, dtype=torch.float32) * std + mean
            theta0 = base.to(dt[cfg.theta0_dtype])
            del base
            theta = theta0.to(torch.float32) + torch.randn(shape, generator=gen, device=device,
                                                           dtype=torch.float32) * cfg.delta_std
        if cfg.sigma_mult is None:
            sig = cfg.sigma_fixed
        else:
            d = (theta - theta0.to(torch.float32)).to(torch.float64)
            sig = cfg.sigma_mult * float(d.std()) if d.numel() > 1 else cfg.sigma_mult * cfg.delta_std
            del d
        inp.theta.append(theta)
        inp.theta0.append(theta0)
        inp.sigmas.append(float(np.float32(sig)))
        if with_grads:
            gscale = 1.0 if cfg.name == "c1" else 1e-2
            g = (torch.randn(shape, generator=gen, device=device, dtype=torch.float32) * gscale)
            inp.grad_sim.append(g.to(dt[cfg.grad_dtype]))
            if cfg.name == "c1":
                inp.grad_theta.append(torch.zeros(shape, device=device, dtype=torch.float32))
            else:
                inp.grad_theta.append(torch.randn(shape, generator=gen, device=device, dtype=torch.float32) * 1e-3)
    inp.settings = static_settings(cfg, inp.sigmas)
    return inp


def make_experts(cfg: Config, n_experts: int, device="cpu"):
    """Seeded inputs of an N-expert merge shaped like `cfg`: theta0 (cfg.theta0_dtype, drawn as in
    make_inputs) and n_experts fine-tuned versions theta0 + N(0, delta_std^2), stored in theta0's
    dtype.  Returns (theta0 list, experts as a list over experts of lists over tensors)."""
    import torch

    dt = {"bf16": torch.bfloat16, "f32": torch.float32}
    gen = torch.Generator(device=device)
    gen.manual_seed(cfg.data_seed + 0xE0)
    theta0s, experts = [], [[] for _ in range(n_experts)]
    for spec in cfg.specs:
        mean, std = _init_std(spec.kind)
        base = torch.randn(spec.shape, generator=gen, device=device, dtype=torch.float32) * std + mean
        t0 = base.to(dt[cfg.theta0_dtype])
        del base
        theta0s.append(t0)
        for j in range(n_experts):
            x = t0.to(torch.float32) + torch.randn(spec.shape, generator=gen, device=device,
                                                   dtype=torch.float32) * cfg.delta_std
            experts[j].append(x.to(dt[cfg.theta0_dtype]))
            del x
    return theta0s, experts
