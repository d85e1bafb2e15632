"""Hilbert order of an H x W token grid, by recursive quadrant construction.

Test infrastructure only (see the package docstring).

The paper reorders the H x W image tokens along a Hilbert curve and caches the
resulting path P_(H,W) per feature-map size (Sec. 3.1, Sec. 3.2). It does not
state the curve's orientation or start corner (its figures are not part of the
text), so this oracle fixes one convention and the library follows it:

  * cells are (x, y) with x = column, y = row; a token's row-major id is
    y * W + x;
  * H_0 = [(0, 0)];
  * H_k = T(H_{k-1})            (lower-left quadrant, transposed)
          ++ H_{k-1} + (0, s)   (upper-left)
          ++ H_{k-1} + (s, s)   (upper-right)
          ++ A(H_{k-1}) + (s, 0)  (lower-right, anti-transposed)
    with s = 2^(k-1), T(x, y) = (y, x), A(x, y) = (s-1-y, s-1-x);
  * so the curve starts at (0, 0) and ends at (2^k - 1, 0).

order[d] = row-major id of the d-th cell on the curve; rank = inverse of order.
Every one of the curve's eight symmetric variants gives the same tile masks for
the Hilbert patterns, because those depend only on 1-D positions.

Grids that are not a 2^k x 2^k square. The paper measures 56 x 56, 96 x 96,
160 x 160 and 128 x 256 grids (Tables 1, 3, 6-8) and says only that each size has
one path, computed once and cached (Sec. 3.2); it does not say how the curve
covers such a grid. Reading used here: take the curve on the smallest 2^k x 2^k
square that contains the grid (same convention, grid at its lower-left corner)
and keep the cells inside the grid, in the curve's order. On a 2^k square this
is the curve itself.
"""
from __future__ import annotations

import numpy as np


def is_pow2(n: int) -> bool:
    return n > 0 and (n & (n - 1)) == 0


def hilbert_cells(k: int) -> np.ndarray:
    """Cells (x, y) of the order-k curve in visiting order, shape [4^k, 2]."""
    if k < 0:
        raise ValueError("k must be >= 0")
    if k == 0:
        return np.zeros((1, 2), dtype=np.int64)
    prev = hilbert_cells(k - 1)
    s = 1 << (k - 1)
    x, y = prev[:, 0], prev[:, 1]
    lower_left = np.stack([y, x], axis=1)                      # T
    upper_left = np.stack([x, y + s], axis=1)
    upper_right = np.stack([x + s, y + s], axis=1)
    lower_right = np.stack([(s - 1 - y) + s, (s - 1 - x)], axis=1)  # A, then + (s, 0)
    return np.concatenate([lower_left, upper_left, upper_right, lower_right], axis=0)


def hilbert_order(H: int, W: int) -> np.ndarray:
    """order[d] = row-major id of the d-th token along the curve (int64, length H*W)."""
    if H < 1 or W < 1:
        raise ValueError("the grid must have at least one row and one column")
    k = (max(H, W) - 1).bit_length()          # smallest 2^k >= max(H, W)
    cells = hilbert_cells(k)
    inside = (cells[:, 0] < W) & (cells[:, 1] < H)
    cells = cells[inside]
    return cells[:, 1] * W + cells[:, 0]


def inverse_permutation(order: np.ndarray) -> np.ndarray:
    """rank[order[d]] = d."""
    order = np.asarray(order, dtype=np.int64)
    rank = np.full(order.shape[0], -1, dtype=np.int64)
    rank[order] = np.arange(order.shape[0], dtype=np.int64)
    if (rank < 0).any():
        raise ValueError("not a permutation")
    return rank


def hilbert_rank(H: int, W: int) -> np.ndarray:
    """rank[t] = Hilbert position of row-major token t."""
    return inverse_permutation(hilbert_order(H, W))
