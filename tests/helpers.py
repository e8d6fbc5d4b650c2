"""Shared helpers of the GPU tests: GPU tensors as host arrays in the oracle's storage conventions."""
import numpy as np
import torch


def host(t):
    """(values, dtype name) of a tensor on the host, flattened: bf16 as its uint16 bit patterns,
    fp32 as a float32 copy."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16).ravel(), "bf16"
    return t.numpy().ravel().copy(), "f32"


def bits(t):
    """The raw bits of a bf16 or fp32 tensor, for bit-exact comparisons."""
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)
