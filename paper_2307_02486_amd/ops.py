"""Python entry points of the dilated-attention forward and backward passes.

`plan`/`dilated_attn`, `plan_bwd`/`dilated_attn_bwd` and `xpos` mirror the
C ABI (dilated_attn_plan / dilated_attn_fwd, dilated_attn_bwd_plan /
dilated_attn_bwd, dilated_attn_xpos): torch supplies device memory and the
stream, every step of the computation runs in the HIP kernels of
libdilated_attn.so.
"""
from __future__ import annotations

import ctypes
import functools
from typing import Sequence, Tuple

import torch

from . import _lib

_DTYPES = {torch.float32: _lib.DA_F32, torch.bfloat16: _lib.DA_BF16}


def _dtype_code(dtype) -> int:
    if dtype not in _DTYPES:
        raise TypeError(f"unsupported dtype {dtype}; use float32 or bfloat16")
    return _DTYPES[dtype]


def _pattern_key(patterns) -> tuple:
    return tuple((int(w), int(r)) for (w, r) in patterns)


@functools.lru_cache(maxsize=256)
def _plan_cached(entry: str, B: int, N: int, H: int, D: int, pats: tuple, causal: int, dtype_code: int,
                 scale: float):
    """One dilated_attn_plan (or _bwd_plan) call per distinct problem: the
    returned dict is shared, callers must not modify it."""
    lib = _lib.load()
    arr, n = _lib.pattern_array(pats)
    info = _lib.PlanInfo()
    rc = getattr(lib, entry)(B, N, H, D, arr, n, causal, dtype_code, scale, ctypes.byref(info))
    if rc != 0:
        raise _lib.DilatedAttnError(rc, lib)
    return {k: getattr(info, k) for k, _ in _lib.PlanInfo._fields_}


@functools.lru_cache(maxsize=256)
def _pattern_array_cached(pats: tuple):
    return _lib.pattern_array(pats)


def plan(B: int, N: int, H: int, D: int, patterns: Sequence[Tuple[int, int]], causal: bool = True,
         dtype=torch.bfloat16, scale: float | None = None) -> dict:
    """Validate a problem and return its workspace size and work counts (host only)."""
    return dict(_plan_cached("dilated_attn_plan", int(B), int(N), int(H), int(D), _pattern_key(patterns),
                             int(bool(causal)), _dtype_code(dtype), float(scale or 0.0)))


def plan_raw(B, N, H, D, patterns, causal, dtype_code, scale):
    """Call dilated_attn_plan with raw integer arguments; return (rc, info dict)."""
    lib = _lib.load()
    arr, n = _lib.pattern_array(patterns)
    info = _lib.PlanInfo()
    rc = lib.dilated_attn_plan(B, N, H, D, arr, n, causal, dtype_code, scale, ctypes.byref(info))
    return rc, {k: getattr(info, k) for k, _ in _lib.PlanInfo._fields_}


def workspace_for(q: torch.Tensor, patterns, causal=True, scale=None) -> torch.Tensor:
    """Allocate (with torch) the device workspace a call on q's shape needs."""
    B, N, H, D = q.shape
    info = _plan_cached("dilated_attn_plan", B, N, H, D, _pattern_key(patterns), int(bool(causal)),
                        _dtype_code(q.dtype), float(scale or 0.0))
    return torch.empty(max(256, int(info["workspace_bytes"])), dtype=torch.uint8, device=q.device)


def _check_like(name: str, t: torch.Tensor, shape, dtype, device):
    if t.shape != tuple(shape) or t.dtype != dtype or t.device != device or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dtype} tensor of shape {tuple(shape)} on {device}")


def _stream_use(stream, owned):
    """Tensors this binding allocated on torch's current stream but handed to
    another stream's kernels: tell the allocator, so that their memory is not
    reused before that stream's work is done."""
    if stream != torch.cuda.current_stream(stream.device):
        for t in owned:
            t.record_stream(stream)


def dilated_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                 patterns: Sequence[Tuple[int, int]], causal: bool = True,
                 scale: float | None = None, out: torch.Tensor | None = None,
                 lse: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                 stream: torch.cuda.Stream | None = None):
    """Dilated-attention forward.  q, k, v: [B, N, H, D] contiguous on the GPU.

    Returns (out [B,N,H,D] in q's dtype, lse [B,H,N] float32).  Work is
    enqueued on `stream` (default: torch's current stream) and not waited for.
    A given out, lse or workspace must be a contiguous tensor of the right
    shape, dtype and device (workspace: uint8, at least the planned size).
    """
    lib = _lib.load()
    if q.device.type != "cuda":
        raise RuntimeError("dilated_attn runs on the GPU only; q must be a device tensor")
    if q.dim() != 4:
        raise ValueError("q, k, v must be [B, N, H, D]")
    for t in (q, k, v):
        if not t.is_contiguous() or t.shape != q.shape or t.dtype != q.dtype or t.device != q.device:
            raise ValueError("q, k, v must be contiguous tensors of the same shape, dtype and device")
    B, N, H, D = q.shape
    pats = _pattern_key(patterns)
    dcode = _dtype_code(q.dtype)
    sc = float(scale or 0.0)
    info = _plan_cached("dilated_attn_plan", B, N, H, D, pats, int(bool(causal)), dcode, sc)
    owned = []
    if out is None:
        out = torch.empty_like(q)
        owned.append(out)
    else:
        _check_like("out", out, q.shape, q.dtype, q.device)
    if lse is None:
        lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
        owned.append(lse)
    else:
        _check_like("lse", lse, (B, H, N), torch.float32, q.device)
    if workspace is None:
        workspace = torch.empty(max(256, int(info["workspace_bytes"])), dtype=torch.uint8, device=q.device)
        owned.append(workspace)
    elif workspace.dtype != torch.uint8 or workspace.device != q.device or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 tensor on q's device")
    if stream is None:
        stream = torch.cuda.current_stream(q.device)
    arr, n = _pattern_array_cached(pats)
    rc = lib.dilated_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(),
                              B, N, H, D, arr, n, int(bool(causal)), dcode, sc,
                              workspace.data_ptr(), workspace.numel(), stream.cuda_stream)
    if rc != 0:
        raise _lib.DilatedAttnError(rc, lib)
    _stream_use(stream, owned)
    return out, lse


class StageTimer:
    """Context manager around dilated_attn_profile_begin/end: HIP event timing
    of the two launches of each call made inside it (on the call's own
    stream).  ms_attention and ms_combine sum the attention and the combine
    stage."""

    def __init__(self, capacity: int = 4096):
        self.capacity = capacity
        self.ms_attention = self.ms_combine = 0.0
        self.calls = 0

    def __enter__(self):
        lib = _lib.load()
        rc = lib.dilated_attn_profile_begin(self.capacity)
        if rc != 0:
            raise _lib.DilatedAttnError(rc, lib)
        return self

    def __exit__(self, *exc):
        lib = _lib.load()
        a, c, n = ctypes.c_double(), ctypes.c_double(), ctypes.c_int64()
        rc = lib.dilated_attn_profile_end(ctypes.byref(a), ctypes.byref(c), ctypes.byref(n))
        if rc != 0 and exc[0] is None:
            raise _lib.DilatedAttnError(rc, lib)
        self.ms_attention, self.ms_combine, self.calls = a.value, c.value, n.value
        return False


def plan_bwd(B: int, N: int, H: int, D: int, patterns: Sequence[Tuple[int, int]], causal: bool = True,
             dtype=torch.bfloat16, scale: float | None = None) -> dict:
    """Validate a backward problem and return its workspace size and work (host only)."""
    return dict(_plan_cached("dilated_attn_bwd_plan", int(B), int(N), int(H), int(D), _pattern_key(patterns),
                             int(bool(causal)), _dtype_code(dtype), float(scale or 0.0)))


def bwd_workspace_for(q: torch.Tensor, patterns, causal=True, scale=None) -> torch.Tensor:
    """Allocate (with torch) the device workspace a backward call on q's shape needs."""
    B, N, H, D = q.shape
    info = plan_bwd(B, N, H, D, patterns, causal, q.dtype, scale)
    return torch.empty(max(256, int(info["workspace_bytes"])), dtype=torch.uint8, device=q.device)


def dilated_attn_bwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, out: torch.Tensor,
                     lse: torch.Tensor, dout: torch.Tensor, patterns: Sequence[Tuple[int, int]],
                     causal: bool = True, scale: float | None = None, dq: torch.Tensor | None = None,
                     dk: torch.Tensor | None = None, dv: torch.Tensor | None = None,
                     workspace: torch.Tensor | None = None, stream: torch.cuda.Stream | None = None):
    """Dilated-attention backward: (dq, dk, dv) given the forward's inputs and
    outputs (out, lse) and dout, all on the GPU, [B, N, H, D] contiguous
    (lse [B, H, N] float32).  Enqueued on `stream` and not waited for.  A
    given dq, dk, dv or workspace must be a contiguous tensor of the right
    shape, dtype and device."""
    lib = _lib.load()
    if q.device.type != "cuda":
        raise RuntimeError("dilated_attn_bwd runs on the GPU only; q must be a device tensor")
    if q.dim() != 4:
        raise ValueError("tensors must be [B, N, H, D]")
    for t in (q, k, v, out, dout):
        if not t.is_contiguous() or t.shape != q.shape or t.dtype != q.dtype or t.device != q.device:
            raise ValueError("q, k, v, out, dout must be contiguous tensors of the same shape, dtype, device")
    B, N, H, D = q.shape
    _check_like("lse", lse, (B, H, N), torch.float32, q.device)
    pats = _pattern_key(patterns)
    dcode = _dtype_code(q.dtype)
    sc = float(scale or 0.0)
    info = _plan_cached("dilated_attn_bwd_plan", B, N, H, D, pats, int(bool(causal)), dcode, sc)
    owned = []
    grads = []
    for name, g in (("dq", dq), ("dk", dk), ("dv", dv)):
        if g is None:
            g = torch.empty_like(q)
            owned.append(g)
        else:
            _check_like(name, g, q.shape, q.dtype, q.device)
        grads.append(g)
    dq, dk, dv = grads
    if workspace is None:
        workspace = torch.empty(max(256, int(info["workspace_bytes"])), dtype=torch.uint8, device=q.device)
        owned.append(workspace)
    elif workspace.dtype != torch.uint8 or workspace.device != q.device or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 tensor on q's device")
    if stream is None:
        stream = torch.cuda.current_stream(q.device)
    arr, n = _pattern_array_cached(pats)
    rc = lib.dilated_attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(),
                              dout.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), B, N, H, D,
                              arr, n, int(bool(causal)), dcode, sc,
                              workspace.data_ptr(), workspace.numel(), stream.cuda_stream)
    if rc != 0:
        raise _lib.DilatedAttnError(rc, lib)
    _stream_use(stream, owned)
    return dq, dk, dv


def xpos(x: torch.Tensor, sign: int, transpose: bool = False, center: int | None = None,
         base: float = 10000.0, gamma: float = 0.4, scale_base: float = 512.0,
         out: torch.Tensor | None = None, stream: torch.cuda.Stream | None = None) -> torch.Tensor:
    """xPos of a [B, N, H, D] query (sign=+1) or key (sign=-1) tensor on the
    GPU, or its transpose (transpose=True, the backward's map); center
    defaults to N // 2.  `out` may be x itself.  Enqueued on `stream`."""
    lib = _lib.load()
    if x.device.type != "cuda":
        raise RuntimeError("xpos runs on the GPU only; x must be a device tensor")
    if x.dim() != 4 or not x.is_contiguous():
        raise ValueError("x must be a contiguous [B, N, H, D] tensor")
    B, N, H, D = x.shape
    out = torch.empty_like(x) if out is None else out
    if out.shape != x.shape or out.dtype != x.dtype or out.device != x.device or not out.is_contiguous():
        raise ValueError("out must be a contiguous tensor like x")
    if stream is None:
        stream = torch.cuda.current_stream(x.device)
    rc = lib.dilated_attn_xpos(x.data_ptr(), out.data_ptr(), B, N, H, D, int(sign), int(bool(transpose)),
                               N // 2 if center is None else int(center), float(base), float(gamma),
                               float(scale_base), _dtype_code(x.dtype), stream.cuda_stream)
    if rc != 0:
        raise _lib.DilatedAttnError(rc, lib)
    return out


def wgrad(dy: torch.Tensor, x: torch.Tensor, out: torch.Tensor | None = None, bias_grad: bool = False,
          stream: torch.cuda.Stream | None = None):
    """dw = dy^T x for bf16 dy [K, M] and x [K, N] on the GPU (M, N multiples
    of 128): the weight gradient of a projection y = x w^T + b.  With
    bias_grad=True returns (dw, db), db = the column sums of dy.  Enqueued on
    `stream`; the float32 workspace comes from torch's caching allocator."""
    lib = _lib.load()
    if dy.device.type != "cuda" or x.device != dy.device:
        raise RuntimeError("wgrad runs on the GPU only; dy and x must be tensors of one device")
    if dy.dim() != 2 or x.dim() != 2 or dy.shape[0] != x.shape[0] or not dy.is_contiguous() \
            or not x.is_contiguous() or x.dtype != dy.dtype:
        raise ValueError("dy [K, M] and x [K, N] must be contiguous 2-D tensors of one dtype")
    K, M = dy.shape
    N = x.shape[1]
    need = ctypes.c_uint64(0)
    rc = lib.dilated_attn_wgrad_workspace(K, M, N, ctypes.byref(need))
    if rc != 0:
        raise _lib.DilatedAttnError(rc, lib)
    out = torch.empty((M, N), dtype=dy.dtype, device=dy.device) if out is None else out
    if out.shape != (M, N) or out.dtype != dy.dtype or out.device != dy.device or not out.is_contiguous():
        raise ValueError("out must be a contiguous [M, N] tensor of dy's dtype")
    ws = torch.empty(max(need.value, 16), dtype=torch.uint8, device=dy.device)
    if stream is None:
        stream = torch.cuda.current_stream(dy.device)
    db = torch.empty((M,), dtype=dy.dtype, device=dy.device) if bias_grad else None
    rc = lib.dilated_attn_wgrad(dy.data_ptr(), x.data_ptr(), out.data_ptr(), db.data_ptr() if bias_grad else None,
                                K, M, N, _dtype_code(dy.dtype), ws.data_ptr(), need.value, stream.cuda_stream)
    if rc != 0:
        raise _lib.DilatedAttnError(rc, lib)
    ws.record_stream(stream)
    return (out, db) if bias_grad else out


def layer_norm(x: torch.Tensor, weight: torch.Tensor, bias: torch.Tensor, eps: float = 1e-5,
               stream: torch.cuda.Stream | None = None):
    """LayerNorm over the last dimension of a contiguous bf16 tensor on the
    GPU (E a multiple of 8, at most 2048).  Returns (y, mean, rstd), the
    statistics float32 per row for layer_norm_bwd."""
    lib = _lib.load()
    if x.device.type != "cuda":
        raise RuntimeError("layer_norm runs on the GPU only; x must be a device tensor")
    if not x.is_contiguous() or not weight.is_contiguous() or not bias.is_contiguous():
        raise ValueError("x, weight and bias must be contiguous")
    if x.dim() == 0 or x.shape[-1] == 0:
        raise ValueError("x must have a non-empty last dimension")
    E = x.shape[-1]
    if weight.shape != (E,) or bias.shape != (E,) or weight.dtype != x.dtype or bias.dtype != x.dtype \
            or weight.device != x.device or bias.device != x.device:
        raise ValueError("weight and bias must be [E] tensors of x's dtype and device")
    rows = x.numel() // E
    y = torch.empty_like(x)
    mean = torch.empty(x.shape[:-1], dtype=torch.float32, device=x.device)
    rstd = torch.empty_like(mean)
    if stream is None:
        stream = torch.cuda.current_stream(x.device)
    rc = lib.dilated_attn_layernorm_fwd(x.data_ptr(), weight.data_ptr(), bias.data_ptr(), y.data_ptr(),
                                        mean.data_ptr(), rstd.data_ptr(), rows, E, float(eps),
                                        _dtype_code(x.dtype), stream.cuda_stream)
    if rc != 0:
        raise _lib.DilatedAttnError(rc, lib)
    return y, mean, rstd


def layer_norm_bwd(dy: torch.Tensor, x: torch.Tensor, weight: torch.Tensor, mean: torch.Tensor,
                   rstd: torch.Tensor, stream: torch.cuda.Stream | None = None):
    """Gradients (dx, dweight, dbias) of layer_norm given its saved mean and
    rstd; the float32 workspace comes from torch's caching allocator."""
    lib = _lib.load()
    if dy.device.type != "cuda" or x.device != dy.device:
        raise RuntimeError("layer_norm_bwd runs on the GPU only")
    if dy.shape != x.shape or dy.dtype != x.dtype or not dy.is_contiguous() or not x.is_contiguous():
        raise ValueError("dy and x must be contiguous tensors of one shape and dtype")
    if x.dim() == 0 or x.shape[-1] == 0:
        raise ValueError("x must have a non-empty last dimension")
    E = x.shape[-1]
    rows = x.numel() // E
    if weight.shape != (E,) or weight.dtype != x.dtype or weight.device != x.device:
        raise ValueError("weight must be an [E] tensor of x's dtype and device")
    if mean.numel() != rows or rstd.numel() != rows or mean.dtype != torch.float32 or rstd.dtype != torch.float32 \
            or not mean.is_contiguous() or not rstd.is_contiguous() or not weight.is_contiguous():
        raise ValueError("mean and rstd must be contiguous float32 tensors of one value per row")
    need = ctypes.c_uint64(0)
    rc = lib.dilated_attn_layernorm_bwd_workspace(rows, E, ctypes.byref(need))
    if rc != 0:
        raise _lib.DilatedAttnError(rc, lib)
    dx = torch.empty_like(x)
    dw = torch.empty((E,), dtype=x.dtype, device=x.device)
    db = torch.empty_like(dw)
    ws = torch.empty(max(need.value, 16), dtype=torch.uint8, device=x.device)
    if stream is None:
        stream = torch.cuda.current_stream(x.device)
    rc = lib.dilated_attn_layernorm_bwd(dy.data_ptr(), x.data_ptr(), weight.data_ptr(), mean.data_ptr(),
                                        rstd.data_ptr(), dx.data_ptr(), dw.data_ptr(), db.data_ptr(), rows, E,
                                        _dtype_code(x.dtype), ws.data_ptr(), need.value, stream.cuda_stream)
    if rc != 0:
        raise _lib.DilatedAttnError(rc, lib)
    ws.record_stream(stream)
    return dx, dw, db
