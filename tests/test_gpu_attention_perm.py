"""GPU parity of the forward with the reordering fused in (hla_attn_fwd_perm).

The fused path runs the same arithmetic on the same rows as gather -> attention
-> scatter, so it must agree with that composition bit for bit, for any
permutation; it is also checked against the oracle (dense masked attention in
float64) at the bars of the plain forward: out max-abs <= 2e-2 (bf16) / 1e-4
(fp32), log-sum-exp max-abs <= 1e-3.
"""
import numpy as np
import pytest
import torch

import paper_2511_05832_amd as hla
import workloads as W
from conftest import Pat
from helpers import DEV, TOL_LSE, TOL_OUT, max_abs, np64, sample_rows
from oracle import attention as o_attn
from oracle import hilbert as o_hil
from oracle import permute as o_perm

pytestmark = pytest.mark.gpu


def composed(q, k, v, order, mask, scale):
    """gather -> hla_attn_fwd -> scatter (out and lse back to grid order)."""
    qh, kh, vh = (hla.gather(t, order) for t in (q, k, v))
    out_h, lse_h = hla.attn_fwd(qh, kh, vh, mask, scale)
    out = hla.scatter(out_h, order)
    lse = torch.empty_like(lse_h)
    lse[:, :, order.long()] = lse_h
    return out, lse


def fused_vs_composed(pattern, q, k, v, order, tile_m, scale):
    qd, kd, vd = (t.to(DEV) for t in (q, k, v))
    od = order.to(DEV)
    mask = hla.build_block_mask(pattern, tile_m, 64)
    out_f, lse_f = hla.attn_fwd_perm(qd, kd, vd, od, mask, scale)
    out_c, lse_c = composed(qd, kd, vd, od, mask, scale)
    torch.cuda.synchronize()
    assert torch.equal(out_f, out_c), "out differs from gather -> attention -> scatter"
    assert torch.equal(lse_f, lse_c), "lse differs from gather -> attention -> scatter"
    return out_f.cpu(), lse_f.cpu()


def oracle_grid_order(pattern, q, k, v, order, scale, rows=None):
    """Oracle results in grid order for sequence-position rows `rows` (all if None):
    gather with `order`, attend, and report which grid rows the results belong to."""
    qn, kn, vn = (o_perm.gather(np64(t), order) for t in (q, k, v))
    out, lse = o_attn.attention(qn, kn, vn, pattern, scale, rows=rows)
    grid_rows = order if rows is None else order[rows]
    return out, lse, grid_rows


def perm_cases(n):
    rng = np.random.default_rng(4242)
    kinds = list(hla.PATTERN_IDS)
    cases = []
    for i in range(n):
        kind = kinds[i % len(kinds)]
        dtype = "bf16" if i % 3 else "f32"
        d = int(rng.choice([32, 64]))
        tm = int(rng.choice([64, 128]))
        H, Wd = int(rng.choice([16, 32])), int(rng.choice([16, 32, 48]))
        N = H * Wd
        if N % tm:
            tm = 64
        p0 = {"hilbert_window": int(rng.choice([1, 64, 100, N])),
              "hilbert_slide": int(rng.choice([0, 7, 128, N])),
              "hilbert_neighborhood": int(rng.choice([1, 49, min(N, 300)])),
              "hilbert_shifted_window": int(rng.choice([16, 64, 100])),
              "rowmajor_window": int(rng.choice([1, 4, 7])),
              "rowmajor_slide": int(rng.choice([0, 1, 3])),
              "rowmajor_neighborhood": int(rng.choice([1, 3, 7]))}[kind]
        p1 = 0
        if kind == "hilbert_shifted_window":
            p1 = int(rng.integers(0, p0))
        elif kind == "rowmajor_window":
            p1 = int(rng.choice([2, 5, 16]))
        elif kind == "rowmajor_slide":
            p1 = int(rng.choice([0, 2, 4]))
        elif kind == "rowmajor_neighborhood":
            p1 = int(rng.choice([1, 3, 5]))
        cases.append((Pat(kind, H, Wd, p0, p1), int(rng.integers(1, 3)), int(rng.integers(1, 4)),
                      d, dtype, tm, 3000 + i))
    return cases


@pytest.mark.parametrize("pat,B,Hh,d,dtype,tm,seed", perm_cases(21),
                         ids=lambda x: str(x) if isinstance(x, (Pat, str)) else None)
def test_random_permutation_every_row(pat, B, Hh, d, dtype, tm, seed):
    """Any permutation: bit-identical to the composition, every row within the bars."""
    q, k, v = W.attn_inputs(B, Hh, pat.N, d, dtype, seed)
    order = torch.randperm(pat.N, generator=torch.Generator().manual_seed(seed)).to(torch.int32)
    scale = 1.0 / d ** 0.5
    out, lse = fused_vs_composed(pat, q, k, v, order, tm, scale)
    ref_out, ref_lse, grid_rows = oracle_grid_order(pat, q, k, v, order.numpy(), scale)
    e_out = max_abs(np64(out)[:, :, grid_rows], ref_out)
    e_lse = max_abs(np64(lse)[:, :, grid_rows], ref_lse)
    print(f"{pat} {dtype} d={d} tm={tm}: out err {e_out:.3e}, lse err {e_lse:.3e}")
    assert e_out <= TOL_OUT[dtype] and e_lse <= TOL_LSE, (e_out, e_lse)


@pytest.mark.parametrize("w", [W.C1, W.C2, W.C3, W.C4], ids=lambda w: w.name)
def test_workloads_with_the_hilbert_order(w):
    """The measured workloads in their launch configuration, with the Hilbert order
    the library computes: bit-identical to the composition; sampled rows (all rows
    for the small ones) against the oracle."""
    q, k, v = W.workload_inputs(w)
    order, _ = hla.hilbert_perm(w.pattern.H, w.pattern.W)
    out, lse = fused_vs_composed(w.pattern, q, k, v, order.cpu(), w.tile_m, w.scale)
    rows = None if w.N * w.B * w.heads <= 1 << 15 else sample_rows(w.N, w.tile_m, w.seed, 96)
    ref_order = o_hil.hilbert_order(w.pattern.H, w.pattern.W)
    ref_out, ref_lse, grid_rows = oracle_grid_order(w.pattern, q, k, v, ref_order, w.scale, rows)
    e_out = max_abs(np64(out)[:, :, grid_rows], ref_out)
    e_lse = max_abs(np64(lse)[:, :, grid_rows], ref_lse)
    print(f"{w.name}: out err {e_out:.3e}, lse err {e_lse:.3e}")
    assert e_out <= TOL_OUT[w.dtype] and e_lse <= TOL_LSE, (e_out, e_lse)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_identity_order_equals_plain_forward(dtype):
    pat = Pat("hilbert_slide", 32, 32, 90)
    q, k, v = (t.to(DEV) for t in W.attn_inputs(2, 2, pat.N, 64, dtype, 31))
    mask = hla.build_block_mask(pat, 128, 64)
    ident = torch.arange(pat.N, dtype=torch.int32, device=DEV)
    out_f, lse_f = hla.attn_fwd_perm(q, k, v, ident, mask, 0.125)
    out_p, lse_p = hla.attn_fwd(q, k, v, mask, 0.125)
    torch.cuda.synchronize()
    assert torch.equal(out_f, out_p) and torch.equal(lse_f, lse_p)


def test_rejects_wrong_order_length():
    pat = Pat("hilbert_window", 16, 16, 64)
    q, k, v = (t.to(DEV) for t in W.attn_inputs(1, 1, pat.N, 64, "bf16", 1))
    mask = hla.build_block_mask(pat, 64, 64)
    with pytest.raises(hla.HLAError):
        hla.attn_fwd_perm(q, k, v, torch.arange(pat.N - 1, dtype=torch.int32, device=DEV), mask)
