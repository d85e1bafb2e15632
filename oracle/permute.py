"""Gather into and scatter out of Hilbert order (the paper's "reshape" step).

Test infrastructure only (see the package docstring).

The paper's input processing reorders the tokens with the cached path before
the QKV projection (Sec. 4.2, input-processing paragraph; Tables 8 and 10,
"Reshape" column). For a tensor with tokens on axis -2:

  gather:  Xh[..., i, :] = X[..., order[i], :]
  scatter: Y[..., order[i], :] = Yh[..., i, :]
"""
from __future__ import annotations

import numpy as np


def gather(x: np.ndarray, order: np.ndarray) -> np.ndarray:
    return np.asarray(x)[..., np.asarray(order, dtype=np.int64), :]


def scatter(xh: np.ndarray, order: np.ndarray) -> np.ndarray:
    xh = np.asarray(xh)
    out = np.empty_like(xh)
    out[..., np.asarray(order, dtype=np.int64), :] = xh
    return out
