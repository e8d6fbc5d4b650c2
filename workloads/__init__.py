"""Seeded synthetic inputs shared by the HIP path's tests/bench and the CPU oracle's tests."""
from .configs import (ALL, Config, Inputs, TensorSettings, TensorSpec, config, make_experts, make_inputs,
                      static_settings, step_params, step_scales)

__all__ = ["ALL", "Config", "Inputs", "TensorSettings", "TensorSpec", "config", "make_experts", "make_inputs",
           "static_settings", "step_params", "step_scales"]
