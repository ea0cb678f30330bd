"""MI355X (gfx950) dilated attention, forward and backward passes (LongNet,
Sec. 2.2-2.3).

The computation runs in the HIP kernels of libdilated_attn.so behind the C
ABI declared in include/dilated_attn.h; this package only marshals arguments.
"""
from .ops import (StageTimer, bwd_workspace_for, dilated_attn, dilated_attn_bwd, layer_norm,  # noqa: F401
                  layer_norm_bwd, plan, plan_bwd, plan_raw, wgrad, workspace_for, xpos)
from ._lib import DilatedAttnError, LIB_PATH  # noqa: F401

__all__ = ["StageTimer", "dilated_attn", "dilated_attn_bwd", "plan", "plan_bwd", "plan_raw",
           "workspace_for", "bwd_workspace_for", "xpos", "wgrad", "layer_norm", "layer_norm_bwd", "DilatedAttnError", "LIB_PATH"]
