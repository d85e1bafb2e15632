"""GPU parity on ragged tilings: N not a multiple of the tile sizes (the paper's
56 x 56 grid at block 128, Tables 3 and 6, and small odd grids down to a single
tile that is mostly padding).

Tile lists are bit-exact against the oracle, whose reading is: ceil(N / b)
tiles per axis, padded slots never allowed, an edge tile never full. The
attention forward (plain, reordering fused, position bias) and the backward are
checked against the oracle's float64 results at the usual bars, and every
output buffer sits at the front of a larger sentinel-filled allocation, so a
write past the end of the sequence would show.
"""
import numpy as np
import pytest
import torch

import paper_2511_05832_amd as hla
import workloads as W
from conftest import Pat
from helpers import DEV, TOL_LSE, TOL_OUT, assert_mask_matches_oracle, max_abs, np64
from oracle import attention as o_attn
from oracle import blockmask as o_bm
from oracle import hilbert as o_hil
from oracle import permute as o_perm

pytestmark = pytest.mark.gpu

SENTINEL = 7.0
PAD = 4096   # sentinel elements after each output


def padded(shape, dtype):
    """A tensor of `shape` at the front of a sentinel-filled buffer; returns (view, tail)."""
    n = int(np.prod(shape))
    buf = torch.full((n + PAD,), SENTINEL, dtype=dtype, device=DEV)
    return buf[:n].view(shape), buf[n:]


def assert_tail_untouched(tail, name):
    torch.cuda.synchronize()
    assert bool((tail == SENTINEL).all()), f"{name}: written past its end"


TDT = {"bf16": torch.bfloat16, "f32": torch.float32}

# The paper's 56 x 56 rows (Tables 3 and 6: K = 7 and W = 7) at tile 128 x 64, and
# odd grids whose N is not a multiple of 4 or even of 8.
PAPER_56 = [Pat("hilbert_slide", 56, 56, 24), Pat("hilbert_neighborhood", 56, 56, 49),
            Pat("hilbert_window", 56, 56, 49), Pat("rowmajor_window", 56, 56, 7, 7),
            Pat("rowmajor_slide", 56, 56, 3, 3), Pat("rowmajor_neighborhood", 56, 56, 7, 7)]
ODD = [(Pat("hilbert_slide", 7, 9, 10), 64, "bf16", 64),        # N = 63: one tile, one padded slot
       (Pat("hilbert_window", 5, 13, 16), 128, "bf16", 32),     # N = 65
       (Pat("rowmajor_slide", 9, 15, 2, 3), 128, "f32", 64),    # N = 135
       (Pat("hilbert_neighborhood", 11, 11, 25), 64, "f32", 32),  # N = 121
       (Pat("rowmajor_window", 13, 10, 4, 3), 64, "bf16", 64),  # N = 130
       (Pat("hilbert_shifted_window", 9, 21, 40, 17), 128, "bf16", 64),  # N = 189
       (Pat("hilbert_slide", 1, 1, 0), 64, "bf16", 64),              # N = 1
       (Pat("rowmajor_window", 1, 2, 1, 2), 128, "f32", 32)]         # N = 2


def ragged_random(n):
    rng = np.random.default_rng(5150)
    kinds = list(hla.PATTERN_IDS)
    out = []
    for i in range(n):
        kind = kinds[i % len(kinds)]
        H, Wd = int(rng.integers(3, 40)), int(rng.integers(3, 40))
        N = H * Wd
        p = {"hilbert_window": (int(rng.integers(1, N + 10)), 0),
             "hilbert_slide": (int(rng.integers(0, N)), 0),
             "hilbert_neighborhood": (int(rng.integers(1, N + 1)), 0),
             "rowmajor_window": (int(rng.integers(1, H + 2)), int(rng.integers(1, Wd + 2))),
             "rowmajor_slide": (int(rng.integers(0, H)), int(rng.integers(0, Wd))),
             "rowmajor_neighborhood": (int(rng.integers(1, H + 1)), int(rng.integers(1, Wd + 1)))}
        if kind == "hilbert_shifted_window":
            w = int(rng.integers(1, 100))
            p0, p1 = w, int(rng.integers(0, w))
        else:
            p0, p1 = p[kind]
        out.append((Pat(kind, H, Wd, p0, p1), int(rng.choice([16, 32, 64, 128])),
                    int(rng.choice([16, 32, 64, 128]))))
    return out


@pytest.mark.parametrize("pat,tm,tn", ragged_random(40) + [(p, 128, 64) for p in PAPER_56],
                         ids=lambda x: repr(x) if isinstance(x, Pat) else str(x))
def test_ragged_masks_bit_exact(pat, tm, tn):
    mask = hla.build_block_mask(pat, tm, tn)
    assert (mask.n_qtiles, mask.n_ktiles) == (-(-pat.N // tm), -(-pat.N // tn))
    assert_mask_matches_oracle(mask, pat, tm, tn)


@pytest.mark.parametrize("pat", PAPER_56, ids=repr)
def test_ragged_transposed_lists(pat):
    mask = hla.build_block_mask(pat, 128, 64, columns=True)
    torch.cuda.synchronize()
    ref = o_bm.column_lists(o_bm.classify(pat, 128, 64))
    np.testing.assert_array_equal(mask.n_full_t.cpu().numpy(), ref.n_full)
    np.testing.assert_array_equal(mask.n_part_t.cpu().numpy(), ref.n_part)
    np.testing.assert_array_equal(mask.full_idx_t.cpu().numpy(), ref.full_idx)
    np.testing.assert_array_equal(mask.part_idx_t.cpu().numpy(), ref.part_idx)


def inputs_in_sequence_order(pat, B, Hh, d, dtype, seed):
    """CPU q, k, v in row-major order, the same gathered into sequence order on the GPU
    (Hilbert patterns) and by the oracle; and both sides' orders."""
    q, k, v = W.attn_inputs(B, Hh, pat.N, d, dtype, seed)
    if pat.hilbert:
        order = hla.hilbert_perm(pat.H, pat.W)[0]
        order_np = o_hil.hilbert_order(pat.H, pat.W)
        dev = [hla.gather(t.to(DEV), order) for t in (q, k, v)]
        ref = [o_perm.gather(np64(t), order_np) for t in (q, k, v)]
    else:
        order, order_np = None, np.arange(pat.N, dtype=np.int64)
        dev = [t.to(DEV) for t in (q, k, v)]
        ref = [np64(t) for t in (q, k, v)]
    return (q, k, v), dev, ref, order, order_np


def fwd_cases():
    cases = [(p, 128, "bf16", 64) for p in PAPER_56] + ODD
    return cases


@pytest.mark.parametrize("pat,tm,dtype,d", fwd_cases(), ids=lambda x: repr(x) if isinstance(x, Pat) else str(x))
def test_ragged_forward_every_row(pat, tm, dtype, d):
    B, Hh = 2, 2
    _, (qs, ks, vs), (qn, kn, vn), _, _ = inputs_in_sequence_order(pat, B, Hh, d, dtype, 61 + pat.N)
    scale = 1.0 / d ** 0.5
    mask = hla.build_block_mask(pat, tm, 64)
    out, out_tail = padded((B, Hh, pat.N, d), TDT[dtype])
    lse, lse_tail = padded((B, Hh, pat.N), torch.float32)
    hla.attn_fwd(qs, ks, vs, mask, scale, out=out, lse=lse)
    assert_tail_untouched(out_tail, "out")
    assert_tail_untouched(lse_tail, "lse")
    ref_out, ref_lse = o_attn.attention(qn, kn, vn, pat, scale)
    e_out, e_lse = max_abs(np64(out), ref_out), max_abs(np64(lse), ref_lse)
    print(f"{pat} tile {tm} {dtype} d={d}: out err {e_out:.3e}, lse err {e_lse:.3e}")
    assert e_out <= TOL_OUT[dtype] and e_lse <= TOL_LSE, (e_out, e_lse)


@pytest.mark.parametrize("pat,tm,dtype,d", fwd_cases(), ids=lambda x: repr(x) if isinstance(x, Pat) else str(x))
def test_ragged_fused_reordering(pat, tm, dtype, d):
    """hla_attn_fwd_perm on a ragged tiling: bit-identical to gather -> attention ->
    scatter, and within the bars of the oracle."""
    B, Hh = 1, 2
    q, k, v = (t.to(DEV) for t in W.attn_inputs(B, Hh, pat.N, d, dtype, 71 + pat.N))
    order = (hla.hilbert_perm(pat.H, pat.W)[0] if pat.hilbert else
             torch.randperm(pat.N, generator=torch.Generator().manual_seed(pat.N)).to(torch.int32).to(DEV))
    scale = 1.0 / d ** 0.5
    mask = hla.build_block_mask(pat, tm, 64)
    out, out_tail = padded((B, Hh, pat.N, d), TDT[dtype])
    lse, lse_tail = padded((B, Hh, pat.N), torch.float32)
    hla.attn_fwd_perm(q, k, v, order, mask, scale, out=out, lse=lse)
    assert_tail_untouched(out_tail, "out")
    assert_tail_untouched(lse_tail, "lse")
    qh, kh, vh = (hla.gather(t, order) for t in (q, k, v))
    out_h, lse_h = hla.attn_fwd(qh, kh, vh, mask, scale)
    torch.cuda.synchronize()
    assert torch.equal(out, hla.scatter(out_h, order))
    lse_c = torch.empty_like(lse_h)
    lse_c[:, :, order.long()] = lse_h
    assert torch.equal(lse, lse_c)
    order_np = order.cpu().numpy().astype(np.int64)
    ref_out, ref_lse = o_attn.attention(*(o_perm.gather(np64(t), order_np) for t in (q, k, v)), pat, scale)
    e_out = max_abs(np64(out)[:, :, order_np], ref_out)
    e_lse = max_abs(np64(lse)[:, :, order_np], ref_lse)
    assert e_out <= TOL_OUT[dtype] and e_lse <= TOL_LSE, (e_out, e_lse)


@pytest.mark.parametrize("pat,tm,dtype,d", fwd_cases()[::2] + ODD[1::2],
                         ids=lambda x: repr(x) if isinstance(x, Pat) else str(x))
def test_ragged_position_bias(pat, tm, dtype, d):
    B, Hh = 1, 2
    _, (qs, ks, vs), (qn, kn, vn), order, order_np = inputs_in_sequence_order(pat, B, Hh, d, dtype, 81 + pat.N)
    table = torch.randn((Hh, 2 * pat.H - 1, 2 * pat.W - 1), generator=torch.Generator().manual_seed(pat.N))
    scale = 1.0 / d ** 0.5
    mask = hla.build_block_mask(pat, tm, 64)
    out, out_tail = padded((B, Hh, pat.N, d), TDT[dtype])
    lse, lse_tail = padded((B, Hh, pat.N), torch.float32)
    hla.attn_fwd_rpb(qs, ks, vs, order, table.to(DEV), mask, scale, out=out, lse=lse)
    assert_tail_untouched(out_tail, "out")
    assert_tail_untouched(lse_tail, "lse")
    ref_out, ref_lse = o_attn.attention(qn, kn, vn, pat, scale, rpb=(table.double().numpy(), order_np))
    e_out, e_lse = max_abs(np64(out), ref_out), max_abs(np64(lse), ref_lse)
    print(f"{pat} tile {tm} {dtype} d={d}: out err {e_out:.3e}, lse err {e_lse:.3e}")
    assert e_out <= TOL_OUT[dtype] and e_lse <= TOL_LSE, (e_out, e_lse)


TOL_GRAD = {"bf16": 2e-2, "f32": 1e-4}


@pytest.mark.parametrize("pat,tm,dtype,d", [(PAPER_56[0], 128, "bf16", 64), (PAPER_56[3], 128, "bf16", 64),
                                            (PAPER_56[5], 64, "f32", 64)] + ODD,
                         ids=lambda x: repr(x) if isinstance(x, Pat) else str(x))
def test_ragged_backward(pat, tm, dtype, d):
    """Gradients on a ragged tiling against the oracle's (bars relative to the
    gradient's size, as in the backward tests); dq, dk, dv written up to N only."""
    B, Hh = 1, 2
    (q, _, _), (qs, ks, vs), (qn, kn, vn), order, order_np = inputs_in_sequence_order(pat, B, Hh, d, dtype, 91 + pat.N)
    g = torch.Generator().manual_seed(pat.N + 1)
    dout_cpu = torch.randn(q.shape, generator=g).to(TDT[dtype])
    gn = np64(dout_cpu)
    if pat.hilbert:
        gd = hla.gather(dout_cpu.to(DEV), order)
        gn = o_perm.gather(gn, order_np)
    else:
        gd = dout_cpu.to(DEV)
    scale = 1.0 / d ** 0.5
    mask = hla.build_block_mask(pat, tm, 64, columns=True)
    out, lse = hla.attn_fwd(qs, ks, vs, mask, scale)
    shape = (B, Hh, pat.N, d)
    (dq, tq), (dk, tk), (dv, tv) = (padded(shape, TDT[dtype]) for _ in range(3))
    hla.attn_bwd(qs, ks, vs, out, gd, lse, mask, scale, dq=dq, dk=dk, dv=dv)
    for t, n in ((tq, "dq"), (tk, "dk"), (tv, "dv")):
        assert_tail_untouched(t, n)
    ref = o_attn.attention_backward(qn, kn, vn, gn, pat, scale)
    for name, got, r in zip(("dq", "dk", "dv"), (dq, dk, dv), ref):
        gscale = max(1.0, float(np.abs(r).max()))
        err = max_abs(np64(got), r)
        print(f"{pat} tile {tm} {dtype} {name}: err {err:.3e} (scale {gscale:.3f})")
        assert err <= TOL_GRAD[dtype] * gscale, (name, err)
