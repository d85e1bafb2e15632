"""GPU parity of the forward with the global relative position bias
(hla_attn_fwd_rpb) against the oracle's dense masked attention with the same
bias, in float64, on the same seeded inputs and tables.

Bars as for the plain forward: out max-abs <= 2e-2 (bf16) / 1e-4 (fp32),
log-sum-exp max-abs <= 1e-3.
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


def table_for(pat, heads, seed, std=1.0):
    g = torch.Generator().manual_seed(seed)
    return std * torch.randn((heads, 2 * pat.H - 1, 2 * pat.W - 1), generator=g)


def run_and_check(pat, B, Hh, d, dtype, tm, seed, rows=None, table=None):
    q, k, v = W.attn_inputs(B, Hh, pat.N, d, dtype, seed)
    table = table_for(pat, Hh, seed + 1) if table is None else table
    scale = 1.0 / d ** 0.5
    if pat.hilbert:
        order_np = o_hil.hilbert_order(pat.H, pat.W)
        order = hla.hilbert_perm(pat.H, pat.W)[0]
        qs, ks, vs = (hla.gather(t.to(DEV), order) for t in (q, k, v))
        qn, kn, vn = (o_perm.gather(np64(t), order_np) for t in (q, k, v))
    else:
        order_np = np.arange(pat.N, dtype=np.int64)
        order = None
        qs, ks, vs = (t.to(DEV) for t in (q, k, v))
        qn, kn, vn = (np64(t) for t in (q, k, v))
    mask = hla.build_block_mask(pat, tm, 64)
    out, lse = hla.attn_fwd_rpb(qs, ks, vs, order, table.to(DEV), mask, scale)
    torch.cuda.synchronize()
    ref_out, ref_lse = o_attn.attention(qn, kn, vn, pat, scale, rows=rows,
                                        rpb=(table.double().numpy(), order_np))
    got_out, got_lse = np64(out), np64(lse)
    if rows is not None:
        got_out, got_lse = got_out[:, :, rows], got_lse[:, :, rows]
    e_out, e_lse = max_abs(got_out, ref_out), max_abs(got_lse, ref_lse)
    print(f"{pat} {dtype} d={d} tm={tm}: out err {e_out:.3e}, lse err {e_lse:.3e}")
    assert np.isfinite(got_out).all()
    assert e_out <= TOL_OUT[dtype] and e_lse <= TOL_LSE, (e_out, e_lse)
    return out, lse


CASES = [
    (Pat("hilbert_window", 32, 32, 64), 2, 2, 64, "bf16", 128),
    (Pat("hilbert_slide", 32, 32, 100), 1, 3, 64, "bf16", 64),
    (Pat("hilbert_shifted_window", 32, 32, 64, 32), 1, 2, 32, "bf16", 128),
    (Pat("hilbert_neighborhood", 24, 40, 81), 2, 1, 64, "bf16", 64),
    (Pat("hilbert_slide", 56, 56, 24), 1, 2, 64, "bf16", 64),
    (Pat("rowmajor_window", 32, 32, 8, 8), 1, 2, 64, "bf16", 128),
    (Pat("rowmajor_slide", 16, 48, 3, 3), 2, 1, 32, "bf16", 64),
    (Pat("rowmajor_neighborhood", 32, 16, 5, 5), 1, 2, 64, "bf16", 128),
    (Pat("hilbert_window", 32, 32, 64), 1, 2, 32, "f32", 64),
    (Pat("hilbert_slide", 16, 16, 40), 2, 1, 64, "f32", 128),
    (Pat("rowmajor_slide", 16, 16, 2, 2), 1, 2, 32, "f32", 64),
]


@pytest.mark.parametrize("case", range(len(CASES)), ids=lambda i: f"{CASES[i][0]}-{CASES[i][4]}")
def test_every_row(case):
    pat, B, Hh, d, dtype, tm = CASES[case]
    run_and_check(pat, B, Hh, d, dtype, tm, seed=700 + case)


def test_full_size_window_sampled_rows():
    w = W.C3
    rows = sample_rows(w.N, w.tile_m, w.seed, n_random=64)
    run_and_check(w.pattern, w.B, w.heads, w.d, w.dtype, w.tile_m, 55, rows=rows)


def test_dominant_self_offset_returns_v():
    pat = Pat("hilbert_slide", 32, 32, 50)
    t = torch.zeros((2, 63, 63))
    t[:, 31, 31] = 60.0
    q, k, v = W.attn_inputs(1, 2, pat.N, 64, "bf16", 77)
    order = hla.hilbert_perm(32, 32)[0]
    qs, ks, vs = (hla.gather(x.to(DEV), order) for x in (q, k, v))
    mask = hla.build_block_mask(pat, 128, 64)
    out, _ = hla.attn_fwd_rpb(qs, ks, vs, order, t.to(DEV), mask, 0.125)
    torch.cuda.synchronize()
    assert max_abs(np64(out), np64(vs)) <= 1e-2


def test_rejects_wrong_table_shape():
    pat = Pat("hilbert_window", 16, 16, 64)
    q, k, v = (x.to(DEV) for x in W.attn_inputs(1, 2, pat.N, 64, "bf16", 1))
    mask = hla.build_block_mask(pat, 64, 64)
    with pytest.raises(hla.HLAError):
        hla.attn_fwd_rpb(q, k, v, None, torch.zeros((2, 31, 30), device=DEV), mask)


@pytest.mark.parametrize("H,Wd,dtype", [(32, 32, "bf16"), (8, 8, "bf16"), (16, 24, "f32")], ids=str)
def test_arbitrary_order(H, Wd, dtype):
    """Any order, not just the Hilbert path: with a random permutation the cells of a
    tile scatter over the grid, so a 32 x 32 grid's tile windows (up to 63 x 63
    entries) exceed the staged capacity and the kernel reads the table directly,
    while an 8 x 8 grid keeps staged windows of irregular boxes."""
    pat = Pat("hilbert_slide", H, Wd, 40)
    B, Hh, d = 1, 2, 64
    q, k, v = W.attn_inputs(B, Hh, pat.N, d, dtype, 91)
    g = torch.Generator().manual_seed(H * Wd)
    order = torch.randperm(pat.N, generator=g).to(torch.int32)
    table = torch.randn((Hh, 2 * H - 1, 2 * Wd - 1), generator=g)
    mask = hla.build_block_mask(pat, 128 if pat.N % 128 == 0 else 64, 64)
    scale = 1.0 / d ** 0.5
    out, lse = hla.attn_fwd_rpb(q.to(DEV), k.to(DEV), v.to(DEV), order.to(DEV), table.to(DEV), mask, scale)
    torch.cuda.synchronize()
    ref_out, ref_lse = o_attn.attention(np64(q), np64(k), np64(v), pat, scale,
                                        rpb=(table.double().numpy(), order.numpy().astype(np.int64)))
    e_out, e_lse = max_abs(np64(out), ref_out), max_abs(np64(lse), ref_lse)
    print(f"{H}x{Wd} {dtype}: out err {e_out:.3e}, lse err {e_lse:.3e}")
    assert e_out <= TOL_OUT[dtype] and e_lse <= TOL_LSE, (e_out, e_lse)
