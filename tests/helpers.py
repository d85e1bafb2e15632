"""Shared helpers for the GPU parity tests: run the HIP path through the binding
and evaluate the oracle on the same seeded inputs. The two sides share only the
inputs."""
from __future__ import annotations

import numpy as np
import torch

import paper_2511_05832_amd as hla
from oracle import attention as o_attn
from oracle import blockmask as o_bm
from oracle import hilbert as o_hil
from oracle import permute as o_perm

DEV = "cuda"

# max-abs tolerances for attention outputs and log-sum-exp
TOL_OUT = {"bf16": 2e-2, "f32": 1e-4}
TOL_LSE = 1e-3


def np64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def sample_rows(N: int, tile_m: int, seed: int, n_random: int = 160) -> np.ndarray:
    """Query rows for sampled parity: both sequence ends, the first and last row of a
    spread of query tiles, and random rows."""
    rng = np.random.default_rng(seed)
    n_tiles = N // tile_m
    tiles = np.unique(np.linspace(0, n_tiles - 1, min(n_tiles, 24)).astype(np.int64))
    rows = [0, 1, N - 2, N - 1]
    rows += list(tiles * tile_m) + list(tiles * tile_m + tile_m - 1)
    rows += list(rng.choice(N, size=min(N, n_random), replace=False))
    return np.unique(np.asarray(rows, dtype=np.int64))


def gpu_block_mask_host(mask: hla.BlockMask):
    torch.cuda.synchronize()
    return (mask.n_full.cpu().numpy(), mask.full_idx.cpu().numpy(),
            mask.n_part.cpu().numpy(), mask.part_idx.cpu().numpy())


def assert_mask_matches_oracle(mask: hla.BlockMask, pattern, tile_m, tile_n, qtiles=None):
    nf, fi, npart, pi = gpu_block_mask_host(mask)
    ref = o_bm.build(pattern, tile_m, tile_n, qtiles)
    rows = np.arange(mask.n_qtiles) if qtiles is None else np.asarray(list(qtiles))
    np.testing.assert_array_equal(nf[rows], ref.n_full)
    np.testing.assert_array_equal(npart[rows], ref.n_part)
    np.testing.assert_array_equal(fi[rows], ref.full_idx)
    np.testing.assert_array_equal(pi[rows], ref.part_idx)
    return ref


def _gathers(pattern, gather):
    if gather is None:
        return pattern.kind.startswith("hilbert")
    return gather


def run_hip_attention(pattern, q, k, v, tile_m, tile_n, scale, gather=None):
    """q, k, v: CPU tensors in row-major token order. Hilbert patterns gather them into
    Hilbert order on the GPU first (gather=False: the tensors are taken as already in
    sequence order, for grids that have no Hilbert curve). Returns (out, lse, order) on
    the CPU, in the order the kernel saw."""
    qd, kd, vd = (t.to(DEV) for t in (q, k, v))
    order = None
    if _gathers(pattern, gather):
        order, _ = hla.hilbert_perm(pattern.H, pattern.W)
        qd, kd, vd = (hla.gather(t, order) for t in (qd, kd, vd))
    mask = hla.build_block_mask(pattern, tile_m, tile_n)
    out, lse = hla.attn_fwd(qd, kd, vd, mask, scale)
    torch.cuda.synchronize()
    return out.cpu(), lse.cpu(), (None if order is None else order.cpu().numpy())


def oracle_attention(pattern, q, k, v, scale, rows=None, gather=None):
    """Oracle on the same inputs: Hilbert patterns gather with the oracle's own order."""
    qn, kn, vn = (np64(t) for t in (q, k, v))
    if _gathers(pattern, gather):
        order = o_hil.hilbert_order(pattern.H, pattern.W)
        qn, kn, vn = (o_perm.gather(a, order) for a in (qn, kn, vn))
    return o_attn.attention(qn, kn, vn, pattern, scale, rows=rows)


def max_abs(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    both_inf = np.isinf(a) & np.isinf(b) & (np.sign(a) == np.sign(b))
    d = np.where(both_inf, 0.0, np.abs(a - b))
    return float(np.nan_to_num(d, nan=np.inf).max()) if d.size else 0.0
