"""Dense element-wise-masked softmax attention in float64.

Test infrastructure only (see the package docstring).

For every batch b, head h and query position i, over all key positions j:

  S_ij   = scale * <q_i, k_j>   if mask(i, j) else -inf
  m_i    = max_j S_ij
  l_i    = sum_j exp(S_ij - m_i)
  out_i  = sum_j exp(S_ij - m_i) * v_j / l_i
  lse_i  = m_i + ln(l_i)

This is the result the block-sparse kernel must reproduce: masked entries add
exp(-inf) = 0, empty tiles contribute nothing, and skipping them changes only
the cost (Sec. 3.1 and Eq. 1). The paper checks its block-sparse outputs
against a dense implementation of the same pattern in the same way (Sec. 4.2,
HWT/HNT results). A row with no allowed key (not produced by the paper's
patterns, where every query attends itself) is defined as out = 0,
lse = -inf. The log-sum-exp is natural-log.

Inputs are float arrays [B, heads, N, d] already in the order the pattern's
positions refer to; they are upcast to float64 exactly. ``positions`` maps an
index on the token axis to the pattern position of that token (default:
identity); with positions = Hilbert rank this evaluates a Hilbert pattern on
row-major tensors. ``rows`` restricts the output to those query indices.

Global relative position bias (the score modification of the Hilbert Window
Transformer, Sec. 3.2, and part of the per-block work in Eq. 1): with
``rpb = (table, grid_rows)``, table[h] of shape [2H-1, 2W-1] and grid_rows[i] the
row-major grid id of the token at index i,

  S_ij = scale * <q_i, k_j> + table[h, r_i - r_j + H - 1, c_i - c_j + W - 1]

before the mask, with (r, c) = (grid_rows // W, grid_rows % W). The bias is the
same for every batch element. The paper enlarges the Swin-style window bias to
the whole feature map (its windows have irregular shapes); it gives no table
layout, so the Swin one - offsets shifted to be non-negative, rows then columns
- is used.
"""
from __future__ import annotations

import numpy as np

from . import masks


def rpb_bias(table, grid_rows_q, grid_rows_k, H: int, W: int) -> np.ndarray:
    """Bias [heads, len(q), len(k)] of the global relative position bias: for
    query token at grid id a and key token at grid id b,
    table[h, a//W - b//W + H - 1, a%W - b%W + W - 1]."""
    table = np.asarray(table, dtype=np.float64)
    if table.ndim != 3 or table.shape[1:] != (2 * H - 1, 2 * W - 1):
        raise ValueError(f"table must be [heads, {2 * H - 1}, {2 * W - 1}]")
    a = np.asarray(grid_rows_q, dtype=np.int64)
    b = np.asarray(grid_rows_k, dtype=np.int64)
    dr = a[:, None] // W - b[None, :] // W + H - 1
    dc = a[:, None] % W - b[None, :] % W + W - 1
    return table[:, dr, dc]


def attention(q, k, v, pattern, scale: float, rows=None, positions=None,
              chunk: int = 256, rpb=None):
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, Hh, N, d = q.shape
    if k.shape != (B, Hh, N, d) or v.shape[:3] != (B, Hh, N):
        raise ValueError("q, k, v shapes disagree")
    rows = np.arange(N, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    pos = np.arange(N, dtype=np.int64) if positions is None else np.asarray(positions, dtype=np.int64)
    dv = v.shape[3]
    out = np.zeros((B, Hh, rows.shape[0], dv), dtype=np.float64)
    lse = np.full((B, Hh, rows.shape[0]), -np.inf, dtype=np.float64)
    for c0 in range(0, rows.shape[0], chunk):
        r = rows[c0:c0 + chunk]
        allow = masks.allowed(pattern, pos[r][:, None], pos[None, :])   # [R, N]
        any_allowed = allow.any(axis=1)
        bias = None
        if rpb is not None:
            table, grid_rows = rpb
            grid_rows = np.asarray(grid_rows, dtype=np.int64)
            bias = rpb_bias(table, grid_rows[r], grid_rows, pattern.H, pattern.W)  # [heads, R, N]
        for b in range(B):
            for h in range(Hh):
                s = scale * (q[b, h, r] @ k[b, h].T)                      # [R, N]
                if bias is not None:
                    s = s + bias[h]
                s = np.where(allow, s, -np.inf)
                m = s.max(axis=1)
                m_safe = np.where(any_allowed, m, 0.0)
                p = np.exp(s - m_safe[:, None])
                l = p.sum(axis=1)
                l_safe = np.where(any_allowed, l, 1.0)
                out[b, h, c0:c0 + len(r)] = (p @ v[b, h]) / l_safe[:, None]
                lse[b, h, c0:c0 + len(r)] = np.where(any_allowed, m + np.log(l_safe), -np.inf)
    return out, lse


def attention_backward(q, k, v, dout, pattern, scale: float, rows=None, key_rows=None,
                       positions=None, chunk: int = 256):
    """Gradients of ``attention`` for an upstream gradient ``dout``, in float64.

    The paper times the backward pass of every attention it measures (Tables 1,
    3, 6, 7, 9, 11, Backward columns) but writes no formula for it; the gradients are
    those of the forward definition above. Per (b, h), with P_ij the softmax
    weights (0 where masked) and out_i = sum_j P_ij v_j:

      dv_j  = sum_i P_ij dout_i
      dP_ij = <dout_i, v_j>
      dS_ij = P_ij (dP_ij - sum_j' P_ij' dP_ij')
      dq_i  = scale * sum_j dS_ij k_j
      dk_j  = scale * sum_i dS_ij q_i

    A query with no allowed key has out = 0 whatever the inputs, so it adds
    nothing to any gradient. ``rows`` restricts dq to those query indices and
    ``key_rows`` restricts dk and dv to those key indices; only the queries the
    requested outputs depend on are evaluated (each over all N keys).
    ``positions`` is as in ``attention``. Returns (dq, dk, dv).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    dout = np.asarray(dout, dtype=np.float64)
    B, Hh, N, d = q.shape
    if k.shape != (B, Hh, N, d) or v.shape[:3] != (B, Hh, N) or dout.shape != v.shape:
        raise ValueError("q, k, v, dout shapes disagree")
    pos = np.arange(N, dtype=np.int64) if positions is None else np.asarray(positions, dtype=np.int64)
    rows = np.arange(N, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    keys = np.arange(N, dtype=np.int64) if key_rows is None else np.asarray(key_rows, dtype=np.int64)
    # queries whose softmax rows the requested outputs need
    need = np.zeros(N, dtype=bool)
    need[rows] = True
    if key_rows is None:
        need[:] = True
    else:
        for c0 in range(0, keys.shape[0], chunk):
            kk = keys[c0:c0 + chunk]
            need |= masks.allowed(pattern, pos[:, None], pos[kk][None, :]).any(axis=1)
    qidx = np.nonzero(need)[0]
    slot_of_row = {int(r): n for n, r in enumerate(rows)}
    dv_ = v.shape[3]
    dq = np.zeros((B, Hh, rows.shape[0], d), dtype=np.float64)
    dk = np.zeros((B, Hh, keys.shape[0], d), dtype=np.float64)
    dv = np.zeros((B, Hh, keys.shape[0], dv_), dtype=np.float64)
    for c0 in range(0, qidx.shape[0], chunk):
        r = qidx[c0:c0 + chunk]
        allow = masks.allowed(pattern, pos[r][:, None], pos[None, :])     # [R, N]
        any_allowed = allow.any(axis=1)
        dst = [slot_of_row.get(int(i), -1) for i in r]
        sel = np.array([t for t, s in enumerate(dst) if s >= 0], dtype=np.int64)
        out_slots = np.array([dst[t] for t in sel], dtype=np.int64)
        for b in range(B):
            for h in range(Hh):
                s = scale * (q[b, h, r] @ k[b, h].T)
                s = np.where(allow, s, -np.inf)
                m = np.where(any_allowed, s.max(axis=1), 0.0)
                e = np.exp(s - m[:, None])
                l = np.where(any_allowed, e.sum(axis=1), 1.0)
                p = e / l[:, None]                                         # softmax, 0 if masked
                dp = dout[b, h, r] @ v[b, h].T                             # [R, N]
                ds = p * (dp - (p * dp).sum(axis=1, keepdims=True))
                if sel.size:
                    dq[b, h, out_slots] = scale * (ds[sel] @ k[b, h])
                dk[b, h] += scale * (ds[:, keys].T @ q[b, h, r])
                dv[b, h] += p[:, keys].T @ dout[b, h, r]
    return dq, dk, dv
