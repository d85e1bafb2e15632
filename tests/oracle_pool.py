"""Evaluates the oracle on row chunks in worker processes, so that the full-size
parity checks (every row of a whole (b, h) slice, every query-tile row of a tile
list) finish in seconds instead of minutes.

The workers are spawned (fresh interpreters, nothing inherited from a process
that has touched the GPU), import only NumPy and ``oracle/``, and never use the
GPU. Each call of the oracle is unchanged: the chunks only split the rows it is
asked for, and every row is still computed over all N keys.
"""
from __future__ import annotations

import multiprocessing as mp
import os
import types

import numpy as np

_STATE = {}


def workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(8, n))


def plain_pattern(p):
    """A pattern record that unpickles without importing the module it came from."""
    return types.SimpleNamespace(kind=p.kind, H=int(p.H), W=int(p.W), p0=int(p.p0), p1=int(p.p1))


def _one_blas_thread():
    try:
        from threadpoolctl import threadpool_limits
        _STATE["limits"] = threadpool_limits(1)
    except ImportError:
        pass


def _init_attention(q, k, v, pattern, scale, positions):
    _one_blas_thread()
    _STATE.update(q=q, k=k, v=v, pattern=pattern, scale=scale, positions=positions)


def _attention_rows(rows):
    from oracle import attention
    s = _STATE
    # 32 query rows per step of the oracle's own chunk loop keeps its [rows, N]
    # temporaries small enough to be reused by the allocator rather than mapped
    # (and page-faulted) afresh for every chunk
    return attention.attention(s["q"], s["k"], s["v"], s["pattern"], s["scale"], rows=rows,
                               positions=s["positions"], chunk=32)


def attention_rows(q, k, v, pattern, scale, rows=None, positions=None, chunk=1024):
    """oracle.attention.attention(q, k, v, pattern, scale, rows, positions), computed in
    chunks of query rows across worker processes. Returns (out, lse)."""
    N = q.shape[2]
    rows = np.arange(N, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    parts = [rows[i:i + chunk] for i in range(0, rows.shape[0], chunk)]
    ctx = mp.get_context("spawn")
    with ctx.Pool(workers(), initializer=_init_attention,
                  initargs=(q, k, v, plain_pattern(pattern), scale, positions)) as pool:
        res = pool.map(_attention_rows, parts)
    return (np.concatenate([r[0] for r in res], axis=2), np.concatenate([r[1] for r in res], axis=2))


def _tile_rows(args):
    from oracle import blockmask
    pattern, tile_m, tile_n, qtiles = args
    bm = blockmask.build(pattern, tile_m, tile_n, qtiles)
    return bm.n_full, bm.full_idx, bm.n_part, bm.part_idx


def tile_lists(pattern, tile_m, tile_n, qtiles, chunk=16):
    """oracle.blockmask.build(pattern, tile_m, tile_n, qtiles) across worker processes.
    Returns (n_full, full_idx, n_part, part_idx) for the requested query-tile rows."""
    qtiles = list(qtiles)
    pat = plain_pattern(pattern)
    parts = [(pat, tile_m, tile_n, qtiles[i:i + chunk]) for i in range(0, len(qtiles), chunk)]
    ctx = mp.get_context("spawn")
    with ctx.Pool(workers(), initializer=_one_blas_thread) as pool:
        res = pool.map(_tile_rows, parts)
    return tuple(np.concatenate([r[i] for r in res], axis=0) for i in range(4))


def _layer_batch(args):
    from oracle import layer
    x, w_qkv, w_proj, H, W, heads, half_width, scale = args
    return layer.hnt_layer(x, w_qkv, w_proj, H, W, heads, half_width, scale)


def layer(x, w_qkv, w_proj, H, W, heads, half_width, scale):
    """oracle.layer.hnt_layer on every row, one batch element per task (the layer acts
    on each batch element independently)."""
    parts = [(x[b:b + 1], w_qkv, w_proj, H, W, heads, half_width, scale) for b in range(x.shape[0])]
    ctx = mp.get_context("spawn")
    with ctx.Pool(workers(), initializer=_one_blas_thread) as pool:
        res = pool.map(_layer_batch, parts)
    return np.concatenate(res, axis=0)
