"""Pins for the oracle's attention layer (oracle.layer.hnt_layer): reorder along
the Hilbert path, QKV projection, 1-D slide attention, merged heads, output
projection (Sec. 3.3; Sec. 4.2).

The oracle never reorders tensors: it evaluates the slide mask on Hilbert
ranks. These tests pin it by routes that do not share that shortcut:
- a half-width that covers the whole sequence leaves no mask at all, so the
  layer is textbook multi-head self-attention (torch's nn.MultiheadAttention
  with the same in- and out-projection weights and no biases);
- the paper's own pipeline written with library calls: gather the tokens into
  Hilbert order, torch's scaled_dot_product_attention with a band of
  half-width h on sequence positions, scatter back, project;
- half-width 0 leaves each token only itself, so the layer is the value
  projection followed by the output projection;
- the rows argument returns exactly those rows of the full result.
"""
import numpy as np
import pytest
import torch

from oracle import hilbert as o_hil
from oracle import layer as o_layer


def _inputs(B, H, W, C, c_out, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((B, H * W, C), generator=g, dtype=torch.float64)
    w_qkv = torch.randn((3 * C, C), generator=g, dtype=torch.float64) / C ** 0.5
    w_proj = torch.randn((c_out, C), generator=g, dtype=torch.float64) / C ** 0.5
    return x, w_qkv, w_proj


@pytest.mark.parametrize("H,W,heads,C", [(4, 4, 2, 16), (6, 5, 4, 32), (8, 8, 1, 8)], ids=str)
def test_full_width_is_multi_head_attention(H, W, heads, C):
    x, w_qkv, w_proj = _inputs(2, H, W, C, C, 11 + H)
    scale = 1.0 / (C // heads) ** 0.5
    y = o_layer.hnt_layer(x.numpy(), w_qkv.numpy(), w_proj.numpy(), H, W, heads, H * W, scale)
    mha = torch.nn.MultiheadAttention(C, heads, bias=False, batch_first=True, dtype=torch.float64)
    with torch.no_grad():
        mha.in_proj_weight.copy_(w_qkv)
        mha.out_proj.weight.copy_(w_proj)
        ref, _ = mha(x, x, x, need_weights=False)
    np.testing.assert_allclose(y, ref.numpy(), rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("H,W,h", [(8, 8, 5), (4, 8, 3), (6, 10, 7), (16, 16, 24)], ids=str)
def test_equals_reorder_band_attention_scatter(H, W, h):
    heads, C, c_out = 2, 16, 24
    x, w_qkv, w_proj = _inputs(1, H, W, C, c_out, 5 * h)
    d = C // heads
    scale = 0.3
    y = o_layer.hnt_layer(x.numpy(), w_qkv.numpy(), w_proj.numpy(), H, W, heads, h, scale)
    order = torch.from_numpy(o_hil.hilbert_order(H, W))     # position i holds token order[i]
    xs = x[:, order]                                         # Hilbert sequence
    q, k, v = (xs @ w_qkv.T).reshape(1, H * W, 3, heads, d).permute(2, 0, 3, 1, 4)
    i = torch.arange(H * W)
    band = (i[:, None] - i[None, :]).abs() <= h
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=band, scale=scale)
    merged = o.permute(0, 2, 1, 3).reshape(1, H * W, C)
    back = torch.empty_like(merged)
    back[:, order] = merged                                  # scatter to row-major tokens
    np.testing.assert_allclose(y, (back @ w_proj.T).numpy(), rtol=1e-10, atol=1e-12)


def test_zero_width_is_value_then_output_projection():
    H, W, heads, C = 8, 4, 4, 32
    x, w_qkv, w_proj = _inputs(2, H, W, C, 16, 3)
    y = o_layer.hnt_layer(x.numpy(), w_qkv.numpy(), w_proj.numpy(), H, W, heads, 0, 0.5)
    ref = x @ w_qkv[2 * C:].T @ w_proj.T
    np.testing.assert_allclose(y, ref.numpy(), rtol=1e-10, atol=1e-12)


def test_rows_subset():
    H, W, heads, C = 8, 8, 2, 16
    x, w_qkv, w_proj = _inputs(2, H, W, C, C, 9)
    args = (x.numpy(), w_qkv.numpy(), w_proj.numpy(), H, W, heads, 6, 0.25)
    full = o_layer.hnt_layer(*args)
    rows = np.array([0, 7, 31, 63, 12])
    part = o_layer.hnt_layer(*args, rows=rows)
    np.testing.assert_allclose(part, full[:, rows], rtol=0, atol=1e-14)
