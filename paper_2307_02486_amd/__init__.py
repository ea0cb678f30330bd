"""MI355X (gfx950) dilated attention, forward pass (LongNet, Sec. 2.2-2.3).

The computation runs in the HIP kernels of libdilated_attn.so behind the C
ABI declared in include/dilated_attn.h; this package only marshals arguments.
"""
from .ops import StageTimer, dilated_attn, plan, plan_raw, workspace_for  # noqa: F401
from ._lib import DilatedAttnError, LIB_PATH  # noqa: F401

__all__ = ["StageTimer", "dilated_attn", "plan", "plan_raw", "workspace_for", "DilatedAttnError", "LIB_PATH"]
