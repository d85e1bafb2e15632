"""GPU parity for the Hilbert-neighbourhood-style layer: gather -> QKV projection ->
Hilbert slide attention -> output projection -> scatter, against the oracle's
row-major formulation (which never reorders the tensors).

Tolerance. The HIP path rounds q, k, v and the attention output to bf16 between
stages (relative error <= 2^-9 each), and the softmax weights to bf16 inside the
attention; the oracle keeps float64 throughout. With weights ~ N(0, 0.02^2) the
layer output is small (std ~ 7e-3, max ~ 4e-2), so the absolute 2e-2 bar alone
would say little: the test also bounds the error relative to the output's
largest magnitude, at 1e-2. Four bf16 roundings in sequence (q/k/v, P, O, y)
each add at most 2^-9 relative to the value rounded, so the accumulated error
stays a few times 2^-9 ~ 2e-3 of max|y|.
"""
import numpy as np
import pytest
import torch

import oracle_pool
import paper_2511_05832_amd as hla
import workloads as W
from helpers import max_abs, np64
from oracle import layer as o_layer

REL_BAR = 1e-2

pytestmark = pytest.mark.gpu


def run_layer(w, x, wq, wp):
    xd, wqd, wpd = x.cuda(), wq.cuda(), wp.cuda()
    order, _ = hla.hilbert_perm(w.H, w.W)
    xh = hla.gather(xd, order)
    q, k, v = hla.qkv_proj(xh, wqd, w.heads)
    mask = hla.build_block_mask(w.pattern, w.tile_m, w.tile_n)
    o, _ = hla.attn_fwd(q, k, v, mask, w.scale, with_lse=False)
    yh = hla.out_proj(o, wpd)
    y = hla.scatter(yh, order)
    torch.cuda.synchronize()
    return y.cpu()


def check_layer(w, pooled=False):
    x, wq, wp = W.layer_inputs(w)
    y = np64(run_layer(w, x, wq, wp))
    args = (np64(x), np64(wq), np64(wp), w.H, w.W, w.heads, w.half_width, w.scale)
    ref = oracle_pool.layer(*args) if pooled else o_layer.hnt_layer(*args)
    err = max_abs(y, ref)
    rel = err / float(np.abs(ref).max())
    print(f"{w.name}: max-abs {err:.3e}, relative to max|ref| {rel:.3e}")
    assert err <= 2e-2
    assert rel <= REL_BAR
    return y


def run_layer_one_launch(w, x, wq, wp):
    """The layer in grid order: QKV projection, the one-launch attention (rows and
    tile lists from the curve, in the kernel), output projection."""
    xd, wqd, wpd = x.cuda(), wq.cuda(), wp.cuda()
    q, k, v = hla.qkv_proj(xd, wqd, w.heads)
    o, _ = hla.attn_fwd_hilbert(q, k, v, w.pattern, w.tile_m, w.tile_n, w.scale, with_lse=False)
    y = hla.out_proj(o, wpd)
    torch.cuda.synchronize()
    return y.cpu()


@pytest.mark.parametrize("name", ["hnt_layer_bf16_64x64_b16_6x32", "small"])
def test_layer_one_launch_equals_the_reordered_layer(name):
    """Same arithmetic on the same rows and tiles: bit for bit the layer with
    separate gather and scatter (itself checked against the oracle above)."""
    w = W.C5 if name != "small" else W.LayerWorkload("small", 16, 16, 3, 2, 32, 20, 64, 64, 11)
    x, wq, wp = W.layer_inputs(w)
    assert torch.equal(run_layer_one_launch(w, x, wq, wp), run_layer(w, x, wq, wp))


def test_layer_full_size_every_row():
    """The whole 64 x 64 layer workload (16 x 4096 tokens x 192 features), every row."""
    check_layer(W.C5, pooled=True)


def test_layer_small_every_row():
    w = W.LayerWorkload("layer_small", H=16, W=16, B=2, heads=3, d=64, half_width=20,
                        tile_m=64, tile_n=64, seed=11)
    check_layer(w)


@pytest.mark.parametrize("heads,d", [(6, 32), (2, 64), (4, 64)])
def test_projections_match_fp64_matmul(heads, d):
    """Each projection alone against a float64 matmul of the same bf16 inputs."""
    g = torch.Generator().manual_seed(heads * 100 + d)
    B, N = 2, 384
    C = heads * d
    x = torch.randn((B, N, C), generator=g).to(torch.bfloat16)
    wq = (torch.randn((3 * C, C), generator=g) * 0.05).to(torch.bfloat16)
    wp = (torch.randn((128, C), generator=g) * 0.05).to(torch.bfloat16)
    q, k, v = hla.qkv_proj(x.cuda(), wq.cuda(), heads)
    y = (x.double() @ wq.double().T).reshape(B, N, 3, heads, d).permute(2, 0, 3, 1, 4)
    for got, ref in zip((q, k, v), y):
        err = max_abs(np64(got), ref.numpy())
        assert err <= 2 ** -8 * float(ref.abs().max()) + 1e-6, err
    o = torch.randn((B, heads, N, d), generator=g).to(torch.bfloat16)
    yo = hla.out_proj(o.cuda(), wp.cuda())
    ref = o.double().permute(0, 2, 1, 3).reshape(B, N, C) @ wp.double().T
    assert max_abs(np64(yo), ref.numpy()) <= 2 ** -8 * float(ref.abs().max()) + 1e-6


def test_projection_ragged_token_count():
    """B*N not a multiple of the 128-token workgroup tile."""
    heads, d, B, N = 2, 32, 3, 100
    C = heads * d
    g = torch.Generator().manual_seed(3)
    x = torch.randn((B, N, C), generator=g).to(torch.bfloat16)
    wq = (torch.randn((3 * C, C), generator=g) * 0.1).to(torch.bfloat16)
    q, k, v = hla.qkv_proj(x.cuda(), wq.cuda(), heads)
    ref = (x.double() @ wq.double().T).reshape(B, N, 3, heads, d).permute(2, 0, 3, 1, 4)
    for got, r in zip((q, k, v), ref):
        assert max_abs(np64(got), r.numpy()) <= 2 ** -8 * float(r.abs().max()) + 1e-6


def test_out_projection_ragged_token_count():
    """The output projection with B*N not a multiple of 128 tokens, at widths that
    take the rows-resident kernel (F = 192, a multiple of 96; K = 64 and 192)."""
    for heads, d, F in ((2, 32, 192), (6, 32, 192)):
        B, N = 3, 100
        C = heads * d
        g = torch.Generator().manual_seed(heads * 7 + F)
        o = torch.randn((B, heads, N, d), generator=g).to(torch.bfloat16)
        wp = (torch.randn((F, C), generator=g) * 0.1).to(torch.bfloat16)
        y = hla.out_proj(o.cuda(), wp.cuda())
        ref = o.double().permute(0, 2, 1, 3).reshape(B, N, C) @ wp.double().T
        assert max_abs(np64(y), ref.numpy()) <= 2 ** -8 * float(ref.abs().max()) + 1e-6


@pytest.mark.parametrize("heads,d,B,N,c_out,kind", [(6, 32, 2, 4096, 192, "hilbert"),   # rows kernel
                                                    (2, 32, 3, 100, 192, "random"),     # ragged tokens
                                                    (4, 64, 2, 256, 128, "random")],    # other kernel
                         ids=str)
def test_projections_with_the_reordering_fused(heads, d, B, N, c_out, kind):
    """hla_qkv_proj_perm equals gather -> hla_qkv_proj, and hla_out_proj_perm equals
    hla_out_proj -> scatter, bit for bit."""
    C = heads * d
    g = torch.Generator().manual_seed(heads * 31 + N)
    x = torch.randn((B, N, C), generator=g).to(torch.bfloat16).cuda()
    wq = (torch.randn((3 * C, C), generator=g) * 0.05).to(torch.bfloat16).cuda()
    wp = (torch.randn((c_out, C), generator=g) * 0.05).to(torch.bfloat16).cuda()
    if kind == "hilbert":
        side = int(round(N ** 0.5))
        order = hla.hilbert_perm(side, side)[0]
    else:
        order = torch.randperm(N, generator=g).to(torch.int32).cuda()
    q, k, v = hla.qkv_proj(x, wq, heads, order=order)
    qc, kc, vc = hla.qkv_proj(hla.gather(x, order), wq, heads)
    o = torch.randn((B, heads, N, d), generator=g).to(torch.bfloat16).cuda()
    y = hla.out_proj(o, wp, order=order)
    yc = hla.scatter(hla.out_proj(o, wp), order)
    torch.cuda.synchronize()
    for got, ref in ((q, qc), (k, kc), (v, vc), (y, yc)):
        assert torch.equal(got, ref)


def test_fused_projections_reject_a_null_order():
    x = torch.zeros((1, 64, 64), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((192, 64), dtype=torch.bfloat16, device="cuda")
    q = torch.zeros((1, 2, 64, 32), dtype=torch.bfloat16, device="cuda")
    lib = hla.lib()
    st = lib.hla_qkv_proj_perm(hla._ptr(x), hla._ptr(w), None, hla._ptr(q), hla._ptr(q), hla._ptr(q),
                               1, 64, 2, 32, None)
    assert st == hla.HLA_ERR_INVALID_ARG
    st = lib.hla_out_proj_perm(hla._ptr(q), hla._ptr(w), None, hla._ptr(x), 1, 64, 2, 32, 64, None)
    assert st == hla.HLA_ERR_INVALID_ARG
