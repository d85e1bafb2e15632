"""GPU parity of the backward pass with the reordering fused in (hla_attn_bwd_perm).

Every tensor stays in grid order and sequence position i is row order[i]. The
kernels run the same arithmetic on the same rows as gather -> hla_attn_bwd ->
scatter, so the two must agree bit for bit, for any permutation (Hilbert path or
random, whole and ragged tilings). Small cases are also checked against the
oracle's float64 gradients at the backward bars (max-abs <= 2e-2 * g for bf16,
1e-4 * g for fp32, g = max(1, max |reference|)).
"""
import numpy as np
import pytest
import torch

import paper_2511_05832_amd as hla
import workloads as W
from conftest import Pat
from helpers import DEV, max_abs, np64
from oracle import attention as o_attn
from oracle import permute as o_perm

pytestmark = pytest.mark.gpu

TOL_GRAD = {"bf16": 2e-2, "f32": 1e-4}
SENTINEL = 7.0


def padded(shape, dtype, pad=4096):
    n = int(np.prod(shape))
    buf = torch.full((n + pad,), SENTINEL, dtype=dtype, device=DEV)
    return buf[:n].view(shape), buf[n:]


def run(pat, B, Hh, d, dtype, tm, seed, order_kind):
    q, k, v = (t.to(DEV) for t in W.attn_inputs(B, Hh, pat.N, d, dtype, seed))
    g = torch.Generator().manual_seed(seed + 1)
    dout = torch.randn(q.shape, generator=g).to(q.dtype).to(DEV)
    if order_kind == "hilbert":
        order = hla.hilbert_perm(pat.H, pat.W)[0]
    else:
        order = torch.randperm(pat.N, generator=g).to(torch.int32).to(DEV)
    mask = hla.build_block_mask(pat, tm, 64, columns=True)
    scale = 1.0 / d ** 0.5
    out, lse = hla.attn_fwd_perm(q, k, v, order, mask, scale)
    (dq, tq), (dk, tk), (dv, tv) = (padded(q.shape, q.dtype) for _ in range(3))
    hla.attn_bwd_perm(q, k, v, out, dout, lse, order, mask, scale, dq=dq, dk=dk, dv=dv)
    # the composition on the same data
    qh, kh, vh, oh, gh = (hla.gather(t, order) for t in (q, k, v, out, dout))
    lse_h = lse[:, :, order.long()].contiguous()
    dqh, dkh, dvh = hla.attn_bwd(qh, kh, vh, oh, gh, lse_h, mask, scale)
    torch.cuda.synchronize()
    for t, n in ((tq, "dq"), (tk, "dk"), (tv, "dv")):
        assert bool((t == SENTINEL).all()), f"{n}: written past its end"
    for name, got, ref_h in (("dq", dq, dqh), ("dk", dk, dkh), ("dv", dv, dvh)):
        assert torch.equal(got, hla.scatter(ref_h, order)), f"{name} differs from gather -> attn_bwd -> scatter"
    return (q, k, v, dout), order, (dq, dk, dv), scale


CASES = [
    (Pat("hilbert_window", 32, 32, 64), 2, 2, 64, "bf16", 128, "hilbert"),
    (Pat("hilbert_slide", 64, 64, 128), 1, 2, 64, "bf16", 128, "hilbert"),
    (Pat("hilbert_neighborhood", 32, 32, 49), 1, 2, 32, "bf16", 64, "hilbert"),
    (Pat("hilbert_shifted_window", 32, 32, 64, 32), 1, 2, 64, "bf16", 64, "random"),
    (Pat("rowmajor_slide", 16, 48, 3, 3), 2, 1, 64, "bf16", 128, "random"),
    (Pat("hilbert_slide", 56, 56, 24), 1, 2, 64, "bf16", 128, "hilbert"),   # ragged at 128
    (Pat("hilbert_window", 9, 21, 40), 1, 2, 32, "bf16", 64, "hilbert"),    # N = 189
    (Pat("hilbert_slide", 32, 32, 100), 1, 2, 64, "f32", 128, "hilbert"),
    (Pat("rowmajor_neighborhood", 13, 10, 5, 3), 2, 1, 32, "f32", 64, "random"),  # N = 130
]


@pytest.mark.parametrize("case", range(len(CASES)),
                         ids=lambda i: f"{CASES[i][0]}-{CASES[i][4]}-tm{CASES[i][5]}-{CASES[i][6]}")
def test_equals_gather_backward_scatter(case):
    pat, B, Hh, d, dtype, tm, kind = CASES[case]
    run(pat, B, Hh, d, dtype, tm, 800 + case, kind)


@pytest.mark.parametrize("case", [0, 3, 6, 8], ids=lambda i: f"{CASES[i][0]}-{CASES[i][4]}")
def test_against_the_oracle(case):
    pat, B, Hh, d, dtype, tm, kind = CASES[case]
    (q, k, v, dout), order, got, scale = run(pat, B, Hh, d, dtype, tm, 900 + case, kind)
    on = order.cpu().numpy().astype(np.int64)
    arrs = [o_perm.gather(np64(t), on) for t in (q, k, v, dout)]
    ref = o_attn.attention_backward(*arrs, pat, scale)
    for name, g_grid, r in zip(("dq", "dk", "dv"), got, ref):
        g_seq = np64(g_grid)[:, :, on]
        gscale = max(1.0, float(np.abs(r).max()))
        err = max_abs(g_seq, r)
        print(f"{pat} {dtype} {name}: err {err:.3e} (scale {gscale:.3f})")
        assert err <= TOL_GRAD[dtype] * gscale, (name, err)


def test_measured_window_workload_bit_exact():
    """The 128 x 128 window workload in its launch configuration."""
    w = W.C3
    run(w.pattern, w.B, w.heads, w.d, w.dtype, w.tile_m, 77, "hilbert")


def test_rejects_wrong_order_length():
    pat = Pat("hilbert_window", 16, 16, 64)
    q = torch.zeros((1, 1, pat.N, 64), dtype=torch.bfloat16, device=DEV)
    lse = torch.zeros((1, 1, pat.N), dtype=torch.float32, device=DEV)
    mask = hla.build_block_mask(pat, 64, 64, columns=True)
    with pytest.raises(hla.HLAError):
        hla.attn_bwd_perm(q, q, q, q, q, lse, torch.arange(pat.N - 1, dtype=torch.int32, device=DEV), mask)


# Several heads per dk/dv workgroup in both launches (the override applies to
# the fused and the plain kernel): head counts that do and do not divide
# B*heads and one above it, ragged and whole tilings, Hilbert and random orders. The fused launch
# must still equal gather -> attn_bwd -> scatter bit for bit, and the plain one
# the one-head launch.
@pytest.mark.parametrize("hpw", [2, 3, 5, 8])
@pytest.mark.parametrize("pat,d,tm,order_kind", [
    (Pat("hilbert_window", 32, 32, 64), 64, 128, "hilbert"),
    (Pat("hilbert_slide", 32, 32, 300), 32, 128, "hilbert"),
    (Pat("rowmajor_slide", 20, 30, 3, 4), 64, 128, "random"),
], ids=str)
def test_heads_per_workgroup(monkeypatch, hpw, pat, d, tm, order_kind):
    monkeypatch.setenv("HLA_ATTN_BWD_HEADS_PER_WORKGROUP", "1")
    _, _, ref, _ = run(pat, 2, 3, d, "bf16", tm, 40 + hpw, order_kind)
    monkeypatch.setenv("HLA_ATTN_BWD_HEADS_PER_WORKGROUP", str(hpw))
    _, _, got, _ = run(pat, 2, 3, d, "bf16", tm, 40 + hpw, order_kind)
    for name, a, b in zip(("dq", "dk", "dv"), got, ref):
        assert torch.equal(a, b), f"{name} differs with {hpw} heads per workgroup"
