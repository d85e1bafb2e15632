"""Tile classification by brute force from the element mask.

Test infrastructure only (see the package docstring).

The N x N score matrix is cut into tiles of tile_m query rows by tile_n key
columns. A tile is full when every element in it is allowed, empty when none
is, and partial otherwise (Sec. 3.1, block types; Fig. 3). Empty tiles are
skipped, full tiles run unmasked, partial tiles need the element mask.

The per-query-tile-row lists hold the key-tile indices of the full and of the
partial tiles in ascending order, padded with -1 to n_ktiles entries.

Ragged tiles (N not a multiple of a tile size; the paper's 56 x 56 grid at
block 128, Tables 3 and 6, is one). The paper does not say how it cuts the
ragged edge. Reading used here: the tile grid is ceil(N / tile_m) x
ceil(N / tile_n), and the sequence is padded to whole tiles with positions that
attend nothing and that nothing attends. A tile is full only when all of its
tile_m * tile_n slots are real and allowed, so a tile reaching past N is never
full; it is empty when none of its slots is allowed. With this reading the
printed sparsity of every 56 x 56 row reproduces (see block_sparsity).
"""
from __future__ import annotations

import dataclasses

import numpy as np

from . import masks

EMPTY, PARTIAL, FULL = 0, 1, 2


@dataclasses.dataclass
class BlockMask:
    cls: np.ndarray        # [n_qtiles, n_ktiles] in {EMPTY, PARTIAL, FULL}
    n_full: np.ndarray     # [n_qtiles] int32
    full_idx: np.ndarray   # [n_qtiles, n_ktiles] int32, ascending, -1 padded
    n_part: np.ndarray     # [n_qtiles] int32
    part_idx: np.ndarray   # [n_qtiles, n_ktiles] int32, ascending, -1 padded

    @property
    def total_full(self) -> int:
        return int(self.n_full.sum())

    @property
    def total_part(self) -> int:
        return int(self.n_part.sum())

    @property
    def empty_fraction(self) -> float:
        return float((self.cls == EMPTY).mean())


def tile_counts(pattern, tile_m: int, tile_n: int, qtiles=None) -> np.ndarray:
    """Number of allowed elements in every tile of the requested query-tile rows."""
    N = int(pattern.H) * int(pattern.W)
    if tile_m < 1 or tile_n < 1:
        raise ValueError("tile sizes must be positive")
    nq, nk = -(-N // tile_m), -(-N // tile_n)
    rows = range(nq) if qtiles is None else list(qtiles)
    cols = np.arange(N, dtype=np.int64)
    out = np.zeros((len(rows), nk), dtype=np.int64)
    for r, qt in enumerate(rows):
        qi = np.arange(qt * tile_m, min(N, (qt + 1) * tile_m), dtype=np.int64)
        m = np.zeros((tile_m, nk * tile_n), dtype=bool)      # padded slots stay False
        m[:len(qi), :N] = masks.allowed(pattern, qi[:, None], cols[None, :])
        out[r] = m.reshape(tile_m, nk, tile_n).sum(axis=(0, 2))
    return out


def classify(pattern, tile_m: int, tile_n: int, qtiles=None) -> np.ndarray:
    counts = tile_counts(pattern, tile_m, tile_n, qtiles)
    cls = np.full(counts.shape, PARTIAL, dtype=np.int8)
    cls[counts == 0] = EMPTY
    cls[counts == tile_m * tile_n] = FULL
    return cls


def lists_from_classes(cls: np.ndarray) -> BlockMask:
    nq, nk = cls.shape
    full_idx = np.full((nq, nk), -1, dtype=np.int32)
    part_idx = np.full((nq, nk), -1, dtype=np.int32)
    n_full = np.zeros(nq, dtype=np.int32)
    n_part = np.zeros(nq, dtype=np.int32)
    for q in range(nq):
        f = np.nonzero(cls[q] == FULL)[0]
        p = np.nonzero(cls[q] == PARTIAL)[0]
        full_idx[q, :len(f)] = f
        part_idx[q, :len(p)] = p
        n_full[q] = len(f)
        n_part[q] = len(p)
    return BlockMask(cls=cls, n_full=n_full, full_idx=full_idx,
                     n_part=n_part, part_idx=part_idx)


def build(pattern, tile_m: int, tile_n: int, qtiles=None) -> BlockMask:
    return lists_from_classes(classify(pattern, tile_m, tile_n, qtiles))


def empty_fraction(pattern, tile_m: int, tile_n: int) -> float:
    return float((classify(pattern, tile_m, tile_n) == EMPTY).mean())


def block_sparsity(pattern, block: int) -> float:
    """The tables' "Sparsity" at block size b: the share of the N x N score matrix
    outside the non-empty b x b blocks, each block counted at its full area b^2,
    i.e. 1 - (non-empty blocks) * b^2 / N^2. When b divides N this is the share of
    empty blocks; on a ragged grid (56 x 56 at b = 128) the padded part of the edge
    blocks is counted too, which is how the printed values come out."""
    N = int(pattern.H) * int(pattern.W)
    cls = classify(pattern, block, block)
    nonempty = int((cls != EMPTY).sum())
    return 1.0 - nonempty * block * block / float(N * N)


def column_lists(cls: np.ndarray) -> BlockMask:
    """Per key-tile column: the query tiles whose tile with it is full / partial,
    ascending, -1 padded (the same lists read down the columns of ``cls``; the
    backward pass walks them to accumulate key and value gradients)."""
    return lists_from_classes(np.ascontiguousarray(cls.T))
