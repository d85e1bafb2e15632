"""Element-wise attention masks (which query may attend which key).

Test infrastructure only (see the package docstring).

A pattern is any object with attributes ``kind``, ``H``, ``W``, ``p0``, ``p1``.
``allowed(pattern, i, j)`` takes integer arrays of query and key sequence
positions (broadcast against each other) and returns a boolean array.

Hilbert patterns act on positions in the Hilbert-ordered sequence (Sec. 3.1:
windows and neighbourhoods are formed on the reordered 1-D sequence).
Row-major patterns act on row-major token ids of the H x W grid; they are the
conventional 2-D baselines the paper compares against (Sec. 3.1, Fig. 3;
Tables 1, 3).

  hilbert_window(w)            floor(i/w) == floor(j/w)
                               (contiguous Hilbert windows, Sec. 3.1-3.2)
  hilbert_slide(h)             |i - j| <= h
                               (band in Hilbert order, Sec. 3.3; borders truncate)
  hilbert_neighborhood(k)      j in [s(i), s(i)+k), s(i) = clamp(i - floor(k/2), 0, N-k)
                               (1-D neighbourhood attention: at the borders the
                               window is repeated, not truncated, Sec. 2.1 on NAT
                               and Sec. 3.3)
  hilbert_shifted_window(w,s)  floor((i+w-s)/w) == floor((j+w-s)/w)
                               (windows moved along the sequence by s; the pairs
                               a cyclic shift would join across the sequence ends
                               are masked, Sec. 3.2)
  rowmajor_window(wh, ww)      same (r div wh, c div ww) cell
  rowmajor_slide(rh, rw)       |r - r'| <= rh and |c - c'| <= rw (borders truncate)
  rowmajor_neighborhood(kh,kw) per axis: r' in [s_r(r), s_r(r)+kh) with
                               s_r(r) = clamp(r - floor(kh/2), 0, H-kh); same for c
                               (NA2D)

A K x K slide kernel corresponds to rowmajor_slide(K//2, K//2) and, with the
same token count, to hilbert_slide((K*K-1)//2); a K x K neighbourhood kernel to
rowmajor_neighborhood(K, K) and hilbert_neighborhood(K*K). These readings
reproduce every sparsity value the paper prints for grids whose token count is
a multiple of the block size (Tables 3, 9, 11).
"""
from __future__ import annotations

import numpy as np


def _clamp_start(i, k, n):
    return np.clip(i - (k // 2), 0, n - k)


def allowed(pattern, i, j) -> np.ndarray:
    i = np.asarray(i, dtype=np.int64)
    j = np.asarray(j, dtype=np.int64)
    kind = pattern.kind
    H, W = int(pattern.H), int(pattern.W)
    N = H * W
    p0, p1 = int(pattern.p0), int(pattern.p1)
    if kind == "hilbert_window":
        return (i // p0) == (j // p0)
    if kind == "hilbert_slide":
        return np.abs(i - j) <= p0
    if kind == "hilbert_neighborhood":
        s = _clamp_start(i, p0, N)
        return (j >= s) & (j < s + p0)
    if kind == "hilbert_shifted_window":
        w, s = p0, p1
        return ((i + w - s) // w) == ((j + w - s) // w)
    r_i, c_i = i // W, i % W
    r_j, c_j = j // W, j % W
    if kind == "rowmajor_window":
        return ((r_i // p0) == (r_j // p0)) & ((c_i // p1) == (c_j // p1))
    if kind == "rowmajor_slide":
        return (np.abs(r_i - r_j) <= p0) & (np.abs(c_i - c_j) <= p1)
    if kind == "rowmajor_neighborhood":
        sr = _clamp_start(r_i, p0, H)
        sc = _clamp_start(c_i, p1, W)
        return (r_j >= sr) & (r_j < sr + p0) & (c_j >= sc) & (c_j < sc + p1)
    raise ValueError(f"unknown pattern kind {kind!r}")


def dense(pattern) -> np.ndarray:
    """The full N x N boolean mask (small N only)."""
    N = int(pattern.H) * int(pattern.W)
    idx = np.arange(N, dtype=np.int64)
    return allowed(pattern, idx[:, None], idx[None, :])
