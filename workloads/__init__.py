"""Seeded synthetic workloads for the dilated-attention forward pass.

This module holds only shapes, pattern lists and random draws.  It contains no
part of the attention arithmetic, so both the CPU oracle (through the tests and
the benchmark) and the GPU path can take their inputs from it without sharing
any of the method's code.

Each workload has the shapes of the paper's settings (Sec. 4.1 for H=12, D=64
and the 2K..32K pattern list; Sec. 2.2 geometric schedules; Sec. 3 for one
device's local share of a long sequence).  The paper's real inputs are the
query/key/value projections of source-code tokens in a trained model; those are
not available, so i.i.d. Gaussian tensors stand in for them.
"""
from __future__ import annotations

import dataclasses
from typing import List, Tuple

import torch

BASE_SEED = 20230705


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    index: int
    B: int
    N: int
    H: int
    D: int
    dtype: str          # "f32" or "bf16"
    sigma: float
    patterns: Tuple[Tuple[int, int], ...]   # (w, r) pairs
    causal: bool = True

    @property
    def seed(self) -> int:
        return BASE_SEED + self.index

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    def describe(self) -> dict:
        return {"workload": self.name, "B": self.B, "N": self.N, "H": self.H,
                "D": self.D, "dtype": self.dtype, "sigma": self.sigma,
                "patterns": [list(p) for p in self.patterns],
                "causal": self.causal}


WORKLOADS: List[Workload] = [
    Workload("tiny_n256_h2_d32_f32", 0, 1, 256, 2, 32, "f32", 1.0,
             ((64, 1), (128, 2), (256, 4))),
    Workload("n8k_b2_h12_d64_3pat", 1, 2, 8192, 12, 64, "bf16", 1.0,
             ((2048, 1), (4096, 2), (8192, 4))),
    Workload("n32k_h12_d64_5pat", 2, 1, 32768, 12, 64, "bf16", 1.0,
             ((2048, 1), (4096, 2), (8192, 4), (16384, 6), (32768, 12))),
    Workload("n256k_h16_d64_8pat_geo", 3, 1, 262144, 16, 64, "bf16", 0.5,
             tuple((2048 * 2 ** i, 2 ** i) for i in range(8))),
    Workload("n1m_h16_d128_6pat", 4, 1, 1048576, 16, 128, "bf16", 1.0,
             ((2048, 1), (8192, 2), (32768, 4), (131072, 8), (524288, 16),
              (1048576, 32))),
]

BY_NAME = {w.name: w for w in WORKLOADS}

# Draws larger than this many elements are made chunk by chunk, each chunk from
# its own seed, so the values do not depend on how much memory one draw may use.
CHUNK = 1 << 24


def _draw(shape, dtype, sigma, seed, tensor_id, device):
    numel = 1
    for s in shape:
        numel *= s
    out = torch.empty(numel, dtype=dtype, device=device)
    nchunks = (numel + CHUNK - 1) // CHUNK
    gen = torch.Generator(device=device)
    for c in range(nchunks):
        lo = c * CHUNK
        hi = min(numel, lo + CHUNK)
        gen.manual_seed((seed * 1000003 + tensor_id * 7919 + c) & ((1 << 63) - 1))
        x = torch.randn(hi - lo, generator=gen, device=device, dtype=torch.float32)
        if sigma != 1.0:
            x.mul_(sigma)
        out[lo:hi] = x.to(dtype)   # round to nearest even for bf16
    return out.view(*shape)


def make_qkv(wl: Workload, device="cpu", seed: int | None = None,
             shape_override: dict | None = None):
    """Return q, k, v of shape [B, N, H, D] in the workload's dtype.

    Values are N(0, sigma^2) rounded to the dtype.  The same (seed, device)
    always gives the same tensors.
    """
    seed = wl.seed if seed is None else seed
    B, N, H, D = wl.B, wl.N, wl.H, wl.D
    if shape_override:
        B = shape_override.get("B", B)
        N = shape_override.get("N", N)
        H = shape_override.get("H", H)
        D = shape_override.get("D", D)
    shape = (B, N, H, D)
    dt = wl.torch_dtype
    return tuple(_draw(shape, dt, wl.sigma, seed, t, device) for t in range(3))


def make_random(shape, dtype=torch.float32, sigma=1.0, seed=0, device="cpu",
                tensor_id=0):
    """A seeded N(0, sigma^2) tensor of any shape, rounded to dtype."""
    return _draw(tuple(shape), dtype, sigma, seed, tensor_id, device)


# Dense-versus-dilated runtime sweep on one device, shaped like the paper's
# runtime experiment (Sec. 3.2): tokens per batch held fixed while N grows from
# 8K, the dense baseline being one pattern (w = N, r = 1), i.e. vanilla causal
# attention through the same kernels, and the dilated variant using the
# experiment's segment lengths on one device, 2048 and N, with dilation rates
# keeping w / r = 2048 (the geometric rule of Sec. 2.2; the experiment does not
# state its rates).  H and D are those of the 1M-token workload.
SWEEP_TOKENS = 1 << 20
SWEEP_N = [8192 << i for i in range(8)]          # 8K .. 1M
SWEEP_H, SWEEP_D = 16, 128


def sweep_configs():
    """[(N, B, dense_patterns, dilated_patterns)] for the sweep."""
    out = []
    for N in SWEEP_N:
        B = SWEEP_TOKENS // N
        out.append((N, B, ((N, 1),), ((2048, 1), (N, N // 2048))))
    return out


def sweep_workload(N: int, variant: str) -> Workload:
    """The sweep's configuration at sequence length N as a Workload
    (variant "dense" or "dilated")."""
    _, B, dense, dilated = {c[0]: c for c in sweep_configs()}[N]
    pats = dense if variant == "dense" else dilated
    index = 100 + SWEEP_N.index(N)
    return Workload(f"sweep_{variant}_n{N}", index, B, N, SWEEP_H, SWEEP_D, "bf16", 1.0, pats)
