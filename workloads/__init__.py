"""Seeded synthetic workloads shared by the tests, the bench and the smoke check.

This module holds the workload table and the seeded input generators only. It
contains none of the method's arithmetic (no Hilbert index, no mask, no
attention), so both the HIP path and the CPU oracle may consume what it makes
without sharing any computation.

Workloads follow the paper's timing setup (Sec. 4.1 and Tables 1-3: random
tensors, 16-bit I/O, head_dim 64, block 128) at the five sizes this library is
measured on. Every tensor is drawn in row-major token order with a CPU
``torch.Generator`` seeded per workload, in float32, and rounded to bfloat16
(round-to-nearest-even, torch's ``.to``) where the workload is bf16.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

import torch

# Pattern names (sequence-position patterns act on Hilbert positions; the
# row-major ones act on row-major token ids of the same grid).
HILBERT_WINDOW = "hilbert_window"
HILBERT_SLIDE = "hilbert_slide"
ROWMAJOR_WINDOW = "rowmajor_window"
ROWMAJOR_SLIDE = "rowmajor_slide"
HILBERT_NEIGHBORHOOD = "hilbert_neighborhood"
ROWMAJOR_NEIGHBORHOOD = "rowmajor_neighborhood"
HILBERT_SHIFTED_WINDOW = "hilbert_shifted_window"

PATTERNS = (HILBERT_WINDOW, HILBERT_SLIDE, ROWMAJOR_WINDOW, ROWMAJOR_SLIDE,
            HILBERT_NEIGHBORHOOD, ROWMAJOR_NEIGHBORHOOD, HILBERT_SHIFTED_WINDOW)


@dataclasses.dataclass(frozen=True)
class Pattern:
    """An attention pattern on an H x W token grid.

    kind   one of PATTERNS
    H, W   grid; N = H * W tokens
    p0, p1 pattern parameters:
        hilbert_window          p0 = window length w (tokens)
        hilbert_slide           p0 = band half-width h
        rowmajor_window         p0, p1 = window rows, window cols
        rowmajor_slide          p0, p1 = radius in rows, radius in cols
        hilbert_neighborhood    p0 = neighbourhood length k (tokens)
        rowmajor_neighborhood   p0, p1 = kernel rows, kernel cols
        hilbert_shifted_window  p0 = window length w, p1 = shift s
    """
    kind: str
    H: int
    W: int
    p0: int
    p1: int = 0

    @property
    def N(self) -> int:
        return self.H * self.W

    @property
    def hilbert(self) -> bool:
        return self.kind.startswith("hilbert")


@dataclasses.dataclass(frozen=True)
class AttnWorkload:
    name: str
    pattern: Pattern
    B: int
    heads: int
    d: int
    dtype: str            # "f32" or "bf16"
    tile_m: int
    tile_n: int
    seed: int
    description: str = ""

    @property
    def N(self) -> int:
        return self.pattern.N

    @property
    def scale(self) -> float:
        return 1.0 / float(self.d) ** 0.5


@dataclasses.dataclass(frozen=True)
class LayerWorkload:
    name: str
    H: int
    W: int
    B: int
    heads: int
    d: int
    half_width: int
    tile_m: int
    tile_n: int
    seed: int
    weight_std: float = 0.02
    description: str = ""

    @property
    def N(self) -> int:
        return self.H * self.W

    @property
    def C(self) -> int:
        return self.heads * self.d

    @property
    def scale(self) -> float:
        return 1.0 / float(self.d) ** 0.5

    @property
    def pattern(self) -> Pattern:
        return Pattern(HILBERT_SLIDE, self.H, self.W, self.half_width)


# The five measured workloads, plus the row-major masks run through the same
# kernel for the empty-tile comparison.
C1 = AttnWorkload("hwa_f32_32x32_w64", Pattern(HILBERT_WINDOW, 32, 32, 64),
                  B=1, heads=1, d=32, dtype="f32", tile_m=64, tile_n=64, seed=0,
                  description="Hilbert window attention, fp32, 32x32 grid, window 64, tile 64x64")
C2 = AttnWorkload("hsa_bf16_64x64_h128", Pattern(HILBERT_SLIDE, 64, 64, 128),
                  B=2, heads=4, d=64, dtype="bf16", tile_m=128, tile_n=64, seed=1,
                  description="Hilbert slide attention, bf16, 64x64 grid, band +-128, tile 128x64")
C3 = AttnWorkload("hwa_bf16_128x128_w256", Pattern(HILBERT_WINDOW, 128, 128, 256),
                  B=4, heads=8, d=64, dtype="bf16", tile_m=128, tile_n=64, seed=2,
                  description="Hilbert window attention, bf16, 128x128 grid, window 256, tile 128x64")
C3_ROWMAJOR = AttnWorkload("wsa_bf16_128x128_16x16", Pattern(ROWMAJOR_WINDOW, 128, 128, 16, 16),
                           B=4, heads=8, d=64, dtype="bf16", tile_m=128, tile_n=64, seed=2,
                           description="row-major 16x16 window, bf16, 128x128 grid, tile 128x64")
C4 = AttnWorkload("hsa_bf16_256x256_h512", Pattern(HILBERT_SLIDE, 256, 256, 512),
                  B=1, heads=8, d=64, dtype="bf16", tile_m=128, tile_n=64, seed=3,
                  description="Hilbert slide attention, bf16, 256x256 grid, band +-512, tile 128x64")
C4_ROWMAJOR = AttnWorkload("sa_bf16_256x256_33x33", Pattern(ROWMAJOR_SLIDE, 256, 256, 16, 16),
                           B=1, heads=8, d=64, dtype="bf16", tile_m=128, tile_n=64, seed=3,
                           description="row-major 33x33 slide, bf16, 256x256 grid, tile 128x64")
# (64 x 64 tiles: the band of half-width 64 then has a full tile on the diagonal
# of every query-tile row, 64 full + 126 partial tiles per (b, h) instead of 126
# partial at 128 x 64, a quarter fewer tile FLOPs; measured 34.5 vs 37.4 us)
C5 = LayerWorkload("hnt_layer_bf16_64x64_b16_6x32", H=64, W=64, B=16, heads=6, d=32,
                   half_width=64, tile_m=64, tile_n=64, seed=4,
                   description="HNT-style layer: gather, QKV, Hilbert slide +-64, proj, scatter; tile 64x64")

ATTN_WORKLOADS = (C1, C2, C3, C3_ROWMAJOR, C4, C4_ROWMAJOR)
WORKLOADS = {w.name: w for w in (C1, C2, C3, C3_ROWMAJOR, C4, C4_ROWMAJOR, C5)}


def _generator(seed: int) -> torch.Generator:
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    return g


def _cast(x: torch.Tensor, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        return x.to(torch.bfloat16)
    if dtype == "f32":
        return x
    raise ValueError(f"unknown dtype {dtype!r}")


def attn_inputs(B: int, heads: int, N: int, d: int, dtype: str, seed: int,
                std: float = 1.0) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """q, k, v ~ N(0, std^2), shape [B, heads, N, d], row-major token order, CPU.

    Drawn in the order q, k, v from one generator, in float32, then rounded to
    the workload dtype.
    """
    g = _generator(seed)
    out = []
    for _ in range(3):
        x = torch.randn((B, heads, N, d), generator=g, dtype=torch.float32)
        if std != 1.0:
            x = x * std
        out.append(_cast(x, dtype))
    return tuple(out)


def workload_inputs(w: AttnWorkload):
    return attn_inputs(w.B, w.heads, w.N, w.d, w.dtype, w.seed)


def layer_inputs(w: LayerWorkload):
    """x [B, N, C] ~ N(0,1); W_qkv [3C, C] and W_proj [C, C] ~ N(0, std^2); bf16, CPU.

    Drawn in the order x, W_qkv, W_proj from one generator.
    """
    g = _generator(w.seed)
    C = w.C
    x = torch.randn((w.B, w.N, C), generator=g, dtype=torch.float32)
    wq = torch.randn((3 * C, C), generator=g, dtype=torch.float32) * w.weight_std
    wp = torch.randn((C, C), generator=g, dtype=torch.float32) * w.weight_std
    return x.to(torch.bfloat16), wq.to(torch.bfloat16), wp.to(torch.bfloat16)


def random_shape_inputs(seed: int, B: int, heads: int, N: int, d: int, dtype: str,
                        std: Optional[float] = None):
    """Small randomized-shape inputs for parity sweeps (same recipe, any shape)."""
    return attn_inputs(B, heads, N, d, dtype, seed, 1.0 if std is None else std)
