"""ctypes view of libdilated_attn.so (the C ABI of include/dilated_attn.h).

Argument marshalling only.  torch is imported first so that the library binds
to the HIP runtime torch already loaded (one runtime per process).
"""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (must be loaded before the HIP library, see above)

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdilated_attn.so")

DA_F32 = 0
DA_BF16 = 1
DA_MAX_PATTERNS = 16
ERRORS = {0: "DA_OK", -1: "DA_EINVAL", -2: "DA_EUNSUPPORTED", -3: "DA_EWORKSPACE",
          -4: "DA_EALIGN", -5: "DA_EHIP", -6: "DA_ETOOLARGE"}
NOALLOC_MAX_BYTES = 128 << 20
CODES = {v: k for k, v in ERRORS.items()}


class Pattern(ctypes.Structure):
    _fields_ = [("w", ctypes.c_int64), ("r", ctypes.c_int64)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("workspace_bytes", ctypes.c_uint64),
                ("num_work_items", ctypes.c_int64),
                ("covered_rows", ctypes.c_int64),
                ("sparse_flops", ctypes.c_double),
                ("bytes_attn", ctypes.c_double),
                ("bytes_combine", ctypes.c_double)]


class DilatedAttnError(RuntimeError):
    def __init__(self, code: int, lib):
        self.code = code
        self.name = ERRORS.get(code, str(code))
        msg = lib.dilated_attn_strerror(code).decode()
        super().__init__(f"{self.name}: {msg}")


_LIB = None


def load():
    """Load the built library; raise if it has not been built."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2307_02486_amd.build` (there is no fallback path)")
    lib = ctypes.CDLL(LIB_PATH)
    i64, f32 = ctypes.c_int64, ctypes.c_float
    lib.dilated_attn_plan.argtypes = [i64, i64, i64, i64, ctypes.POINTER(Pattern), i64, i64, i64,
                                      f32, ctypes.POINTER(PlanInfo)]
    lib.dilated_attn_plan.restype = ctypes.c_int
    vp = ctypes.c_void_p
    lib.dilated_attn_fwd.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, ctypes.POINTER(Pattern),
                                     i64, i64, i64, f32, vp, ctypes.c_uint64, vp]
    lib.dilated_attn_fwd.restype = ctypes.c_int
    lib.dilated_attn_fwd_noalloc.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, ctypes.POINTER(Pattern),
                                             i64, i64, i64, f32, vp]
    lib.dilated_attn_fwd_noalloc.restype = ctypes.c_int
    lib.dilated_attn_bwd_plan.argtypes = lib.dilated_attn_plan.argtypes
    lib.dilated_attn_bwd_plan.restype = ctypes.c_int
    lib.dilated_attn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, i64,
                                     ctypes.POINTER(Pattern), i64, i64, i64, f32, vp, ctypes.c_uint64, vp]
    lib.dilated_attn_bwd.restype = ctypes.c_int
    lib.dilated_attn_xpos.argtypes = [vp, vp, i64, i64, i64, i64, i64, i64, i64, f32, f32, f32, i64, vp]
    lib.dilated_attn_xpos.restype = ctypes.c_int
    lib.dilated_attn_wgrad_workspace.argtypes = [i64, i64, i64, ctypes.POINTER(ctypes.c_uint64)]
    lib.dilated_attn_wgrad_workspace.restype = ctypes.c_int
    lib.dilated_attn_wgrad.argtypes = [vp, vp, vp, vp, i64, i64, i64, i64, vp, ctypes.c_uint64, vp]
    lib.dilated_attn_wgrad.restype = ctypes.c_int
    lib.dilated_attn_layernorm_fwd.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, f32, i64, vp]
    lib.dilated_attn_layernorm_fwd.restype = ctypes.c_int
    lib.dilated_attn_layernorm_bwd_workspace.argtypes = [i64, i64, ctypes.POINTER(ctypes.c_uint64)]
    lib.dilated_attn_layernorm_bwd_workspace.restype = ctypes.c_int
    lib.dilated_attn_layernorm_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, vp, ctypes.c_uint64, vp]
    lib.dilated_attn_layernorm_bwd.restype = ctypes.c_int
    lib.dilated_attn_strerror.argtypes = [ctypes.c_int]
    lib.dilated_attn_strerror.restype = ctypes.c_char_p
    lib.dilated_attn_profile_begin.argtypes = [i64]
    lib.dilated_attn_profile_begin.restype = ctypes.c_int
    lib.dilated_attn_profile_end.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double),
                                             ctypes.POINTER(ctypes.c_int64)]
    lib.dilated_attn_profile_end.restype = ctypes.c_int
    _LIB = lib
    return lib


def pattern_array(patterns):
    pats = list(patterns)
    arr = (Pattern * max(1, len(pats)))()
    for i, (w, r) in enumerate(pats):
        arr[i].w = int(w)
        arr[i].r = int(r)
    return arr, len(pats)
