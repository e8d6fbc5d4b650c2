"""SMAT's per-step Scale/Mask/Perturb parameter transform on MI355X (gfx950).

`libsmat.so` (C ABI in include/smat.h) holds the HIP kernels; this package binds it with
ctypes.  Build it with `python -m paper_2609_33437_amd.build`.
"""
from ._lib import (EXPORTS, OP_PARAMS_DTYPE, SMAT_BF16, SMAT_EXPERT, SMAT_F32, SMAT_NOISE_GAUSSIAN,
                   SMAT_NOISE_LAPLACE, SMAT_NOISE_UNIFORM, SMAT_SIMULATED, AdamStepState, MergePlan, Plan, SmatError,
                   StepState, adamw_params, lib, load_library, merge_term, op_params, op_params_array, rng_key,
                   scale_draw, smat_adamw_fused, smat_backward_accum, smat_debug_draws, smat_merge, smat_simulate,
                   smat_stream_copy)

__all__ = ["EXPORTS", "OP_PARAMS_DTYPE", "op_params_array", "SMAT_BF16", "SMAT_EXPERT", "SMAT_F32", "SMAT_NOISE_GAUSSIAN", "SMAT_NOISE_LAPLACE", "SMAT_NOISE_UNIFORM",
           "SMAT_SIMULATED", "MergePlan", "Plan", "SmatError", "StepState", "AdamStepState", "adamw_params", "lib", "load_library", "merge_term",
           "op_params", "rng_key", "scale_draw", "smat_adamw_fused", "smat_backward_accum", "smat_debug_draws", "smat_merge",
           "smat_simulate", "smat_stream_copy"]
