"""Pins for the oracle's global relative position bias (score modification of the
Hilbert Window Transformer, Sec. 3.2; part of the per-block work in Eq. 1).

The bias table is indexed by the 2-D offset between the query's and the key's
grid cells. These tests fix the index arithmetic by hand-worked examples and the
attention with bias by torch's scaled_dot_product_attention with an additive
float mask, plus the special cases where the bias vanishes, is constant, or
dominates.
"""
import numpy as np
import pytest
import torch

from conftest import Pat
from oracle import attention as o_attn
from oracle import hilbert as o_hil
from oracle import masks


def test_bias_index_by_hand_2x2():
    # table[a][b] = 10a + b, so the entry read names its own (row, col) offset index
    t = np.array([[[0, 1, 2], [10, 11, 12], [20, 21, 22]]], dtype=np.float64)
    ids = np.arange(4)          # row-major cells (0,0), (0,1), (1,0), (1,1)
    got = o_attn.rpb_bias(t, ids, ids, 2, 2)[0]
    want = [[11, 10, 1, 0],
            [12, 11, 2, 1],
            [21, 20, 11, 10],
            [22, 21, 12, 11]]
    assert got.tolist() == want


def test_bias_index_by_hand_single_row():
    t = np.array([[[5.0, 6.0, 7.0, 8.0, 9.0]]])     # H = 1, W = 3: offsets -2..2
    ids = np.arange(3)
    got = o_attn.rpb_bias(t, ids, ids, 1, 3)[0]
    assert got.tolist() == [[7, 6, 5], [8, 7, 6], [9, 8, 7]]


def _inputs(pat, B, Hh, d, seed):
    g = torch.Generator().manual_seed(seed)
    q, k, v = (torch.randn((B, Hh, pat.N, d), generator=g, dtype=torch.float64) for _ in range(3))
    table = torch.randn((Hh, 2 * pat.H - 1, 2 * pat.W - 1), generator=g, dtype=torch.float64)
    return q, k, v, table


@pytest.mark.parametrize("pat", [Pat("hilbert_window", 8, 8, 16), Pat("hilbert_slide", 8, 8, 5),
                                 Pat("rowmajor_window", 6, 8, 2, 4), Pat("hilbert_neighborhood", 8, 4, 9)],
                         ids=str)
def test_matches_sdpa_with_additive_mask(pat):
    q, k, v, table = _inputs(pat, 2, 3, 16, 5)
    grid = (o_hil.hilbert_order(pat.H, pat.W) if pat.hilbert
            else np.arange(pat.N, dtype=np.int64))
    scale = 0.25
    out, lse = o_attn.attention(q.numpy(), k.numpy(), v.numpy(), pat, scale, rpb=(table.numpy(), grid))
    pos = np.arange(pat.N)
    allow = torch.from_numpy(masks.allowed(pat, pos[:, None], pos[None, :]))
    bias = torch.from_numpy(o_attn.rpb_bias(table.numpy(), grid, grid, pat.H, pat.W))  # [heads, N, N]
    add = bias[None].masked_fill(~allow, float("-inf"))
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=add, scale=scale)
    ref_lse = torch.logsumexp(scale * q @ k.transpose(-1, -2) + add, dim=-1)
    np.testing.assert_allclose(out, ref.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(lse, ref_lse.numpy(), rtol=1e-10, atol=1e-12)


def test_zero_table_is_plain_attention():
    pat = Pat("hilbert_slide", 8, 8, 7)
    q, k, v, table = _inputs(pat, 1, 2, 8, 6)
    grid = o_hil.hilbert_order(8, 8)
    a = o_attn.attention(q.numpy(), k.numpy(), v.numpy(), pat, 0.3)
    b = o_attn.attention(q.numpy(), k.numpy(), v.numpy(), pat, 0.3,
                         rpb=(np.zeros_like(table.numpy()), grid))
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_constant_table_shifts_lse_only():
    pat = Pat("hilbert_window", 8, 8, 16)
    q, k, v, table = _inputs(pat, 1, 2, 8, 7)
    grid = o_hil.hilbert_order(8, 8)
    a_out, a_lse = o_attn.attention(q.numpy(), k.numpy(), v.numpy(), pat, 0.3)
    c = 2.5
    b_out, b_lse = o_attn.attention(q.numpy(), k.numpy(), v.numpy(), pat, 0.3,
                                    rpb=(np.full_like(table.numpy(), c), grid))
    np.testing.assert_allclose(b_out, a_out, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(b_lse, a_lse + c, rtol=1e-12, atol=1e-12)


def test_dominant_self_offset_returns_v():
    """A large bias on the zero offset makes every query attend (almost) only itself."""
    pat = Pat("hilbert_slide", 8, 8, 10)
    q, k, v, table = _inputs(pat, 1, 2, 8, 8)
    t = np.zeros_like(table.numpy())
    t[:, pat.H - 1, pat.W - 1] = 80.0
    out, _ = o_attn.attention(q.numpy(), k.numpy(), v.numpy(), pat, 0.1,
                              rpb=(t, o_hil.hilbert_order(8, 8)))
    np.testing.assert_allclose(out, v.numpy(), atol=1e-20 + 1e-12)
