"""A synthetic decoder-only language model and seeded token batches for training-loop runs.

The model is shaped like the Llama decoders SMAT fine-tunes: RMSNorm, multi-head causal
attention, a SwiGLU MLP, and an output layer tied to the token embedding.  Weights are random;
nothing is loaded.  It holds none of SMAT's arithmetic.

Attention scores and their softmax are computed in fp32, outside autocast.  Only the linear
layers run in bf16 under autocast.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import torch
import torch.nn.functional as F
from torch import nn


@dataclass(frozen=True)
class DecoderShape:
    vocab: int
    d: int
    layers: int
    heads: int
    ffn: int


# Llama-3.2-1B-like widths (d 2048, 16 layers, SwiGLU 8192, tied 128256-token embedding), but
# with full multi-head attention: 1.34B parameters.
LLAMA_1B = DecoderShape(vocab=128256, d=2048, layers=16, heads=32, ffn=8192)
TINY = DecoderShape(vocab=96, d=64, layers=2, heads=4, ffn=160)


class RMSNorm(nn.Module):
    def __init__(self, d: int, eps: float = 1e-6):
        super().__init__()
        self.weight = nn.Parameter(torch.ones(d))
        self.eps = eps

    def forward(self, x):
        xf = x.float()
        y = xf * torch.rsqrt(xf.pow(2).mean(-1, keepdim=True) + self.eps)
        return (y * self.weight.float()).to(x.dtype)


class Attention(nn.Module):
    def __init__(self, d: int, heads: int):
        super().__init__()
        self.heads = heads
        self.q_proj = nn.Linear(d, d, bias=False)
        self.k_proj = nn.Linear(d, d, bias=False)
        self.v_proj = nn.Linear(d, d, bias=False)
        self.o_proj = nn.Linear(d, d, bias=False)

    def forward(self, x):
        b, s, d = x.shape
        h, dh = self.heads, d // self.heads

        def split(t):
            return t.view(b, s, h, dh).transpose(1, 2).float().contiguous()

        q, k, v = split(self.q_proj(x)), split(self.k_proj(x)), split(self.v_proj(x))
        with torch.autocast(device_type=x.device.type, enabled=False):
            scores = torch.matmul(q, k.transpose(-1, -2).contiguous()) * (1.0 / math.sqrt(dh))
            causal = torch.ones(s, s, dtype=torch.bool, device=x.device).triu(1)
            p = torch.softmax(scores.masked_fill(causal, float("-inf")), dim=-1)
            o = torch.matmul(p, v)
        o = o.transpose(1, 2).reshape(b, s, d).to(x.dtype)
        return self.o_proj(o)


class MLP(nn.Module):
    def __init__(self, d: int, ffn: int):
        super().__init__()
        self.gate_proj = nn.Linear(d, ffn, bias=False)
        self.up_proj = nn.Linear(d, ffn, bias=False)
        self.down_proj = nn.Linear(ffn, d, bias=False)

    def forward(self, x):
        return self.down_proj(F.silu(self.gate_proj(x)) * self.up_proj(x))


class Block(nn.Module):
    def __init__(self, d: int, heads: int, ffn: int):
        super().__init__()
        self.input_norm = RMSNorm(d)
        self.attn = Attention(d, heads)
        self.post_norm = RMSNorm(d)
        self.mlp = MLP(d, ffn)

    def forward(self, x):
        x = x + self.attn(self.input_norm(x))
        return x + self.mlp(self.post_norm(x))


class Decoder(nn.Module):
    def __init__(self, shape: DecoderShape):
        super().__init__()
        self.shape = shape
        self.embed = nn.Embedding(shape.vocab, shape.d)
        self.blocks = nn.ModuleList([Block(shape.d, shape.heads, shape.ffn) for _ in range(shape.layers)])
        self.norm = RMSNorm(shape.d)
        self.lm_head = nn.Linear(shape.d, shape.vocab, bias=False)
        self.lm_head.weight = self.embed.weight

    def forward(self, tokens):
        x = self.embed(tokens)
        if torch.is_autocast_enabled(tokens.device.type):
            x = x.to(torch.get_autocast_dtype(tokens.device.type))
        for blk in self.blocks:
            x = blk(x)
        return self.lm_head(self.norm(x))

    def loss(self, tokens):
        logits = self(tokens[:, :-1])
        return F.cross_entropy(logits.float().reshape(-1, logits.shape[-1]), tokens[:, 1:].reshape(-1))


def make_decoder(shape: DecoderShape, seed: int, device="cpu") -> Decoder:
    """Random-initialised decoder (normal(0, 0.02) linear and embedding weights, unit norms)."""
    g = torch.Generator().manual_seed(seed)
    model = Decoder(shape)
    with torch.no_grad():
        for name, p in model.named_parameters():
            if p.dim() >= 2:
                p.copy_(torch.randn(p.shape, generator=g) * 0.02)
    return model.to(device)


def token_batches(shape: DecoderShape, batch: int, seq: int, count: int, seed: int, device="cpu"):
    """`count` seeded batches of uniformly drawn token ids, [batch, seq + 1] each."""
    g = torch.Generator().manual_seed(seed)
    return [torch.randint(0, shape.vocab, (batch, seq + 1), generator=g).to(device) for _ in range(count)]


def parameter_count(shape: DecoderShape) -> int:
    d, f = shape.d, shape.ffn
    return shape.vocab * d + shape.layers * (4 * d * d + 3 * d * f + 2 * d) + d
