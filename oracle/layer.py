"""Hilbert-neighbourhood-style attention layer, computed in row-major order.

Test infrastructure only (see the package docstring).

The paper's layer pipeline is: reorder the tokens along the cached Hilbert
path, project to Q, K, V with one linear layer, run the 1-D local attention on
the reordered sequence, and project the merged heads (Sec. 3.3; Sec. 4.2,
input-processing paragraph; Tables 8 and 10). Because the projections act on
each token independently, the same result is obtained without ever reordering
the tensors: evaluate the slide mask on Hilbert positions,

  mask(t, u) = |rank[t] - rank[u]| <= h,

with t, u row-major token ids. This oracle does exactly that, so it shares no
reordering step with the library's gather / scatter path.

Readings where the paper is silent: the QKV projection has no bias; its output
features are laid out as [q | k | v], each block head-major with head_dim
contiguous (reshape (B, N, 3, heads, d)); the output projection has no bias.
"""
from __future__ import annotations

import numpy as np

from . import attention as attn_mod
from . import hilbert


class _Slide:
    def __init__(self, H, W, h):
        self.kind, self.H, self.W, self.p0, self.p1 = "hilbert_slide", H, W, h, 0


def hnt_layer(x, w_qkv, w_proj, H: int, W: int, heads: int, half_width: int,
              scale: float, rows=None):
    """x [B, N, C] row-major tokens; w_qkv [3C, C]; w_proj [C_out, C].

    Returns y [B, N or len(rows), C_out] in row-major token order.
    """
    x = np.asarray(x, dtype=np.float64)
    w_qkv = np.asarray(w_qkv, dtype=np.float64)
    w_proj = np.asarray(w_proj, dtype=np.float64)
    B, N, C = x.shape
    d = C // heads
    rank = hilbert.hilbert_rank(H, W)
    qkv = x @ w_qkv.T                                        # [B, N, 3C]
    qkv = qkv.reshape(B, N, 3, heads, d).transpose(2, 0, 3, 1, 4)  # [3, B, heads, N, d]
    q, k, v = qkv[0], qkv[1], qkv[2]
    o, _ = attn_mod.attention(q, k, v, _Slide(H, W, half_width), scale,
                              rows=rows, positions=rank)     # [B, heads, R, d]
    R = o.shape[2]
    merged = o.transpose(0, 2, 1, 3).reshape(B, R, C)
    return merged @ w_proj.T
