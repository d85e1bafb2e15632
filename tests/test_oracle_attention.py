"""Pins for the oracle's dense masked attention and the layer pipeline.

Pinned to a library routine (PyTorch's scaled_dot_product_attention in float64
on the CPU, with a boolean mask), to a literal loop on tiny inputs, and to the
special cases that reduce to closed forms: an all-allowed mask is plain softmax
attention; a mask that keeps only the diagonal returns v itself with
lse = scale * <q_i, k_i>; Hilbert attention on gathered tensors equals the same
pattern evaluated on Hilbert positions of the row-major tensors (the paper's
"same pattern, same outputs" check of Sec. 4.2, HWT/HNT results).
"""
import math

import numpy as np
import pytest
import torch

from conftest import Pat
from oracle import attention, hilbert, layer, masks, permute


def rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def sdpa_ref(q, k, v, mask, scale):
    qt, kt, vt = (torch.from_numpy(np.ascontiguousarray(a)) for a in (q, k, v))
    m = torch.from_numpy(mask)
    out = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=m, scale=scale)
    s = (qt @ kt.transpose(-1, -2)) * scale
    s = s.masked_fill(~m, float("-inf"))
    lse = torch.logsumexp(s, dim=-1)
    return out.numpy(), lse.numpy()


PATS = [Pat("hilbert_window", 8, 8, 16), Pat("hilbert_slide", 8, 8, 6),
        Pat("rowmajor_window", 8, 8, 2, 4), Pat("rowmajor_slide", 8, 8, 1, 1),
        Pat("hilbert_neighborhood", 8, 8, 9), Pat("rowmajor_neighborhood", 8, 8, 3, 3),
        Pat("hilbert_shifted_window", 8, 8, 16, 8), Pat("hilbert_window", 16, 16, 64)]


@pytest.mark.parametrize("pat", PATS, ids=repr)
@pytest.mark.parametrize("d", [8, 32])
def test_matches_sdpa(pat, d):
    N = pat.H * pat.W
    q, k, v = (rand((2, 3, N, d), s) for s in (1, 2, 3))
    scale = 1 / math.sqrt(d)
    out, lse = attention.attention(q, k, v, pat, scale, chunk=37)
    ref_out, ref_lse = sdpa_ref(q, k, v, masks.dense(pat), scale)
    np.testing.assert_allclose(out, ref_out, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, ref_lse, rtol=0, atol=1e-12)


def test_literal_loop():
    pat = Pat("rowmajor_slide", 4, 4, 1, 1)
    N, d = 16, 4
    q, k, v = (rand((1, 1, N, d), s) for s in (4, 5, 6))
    scale = 0.37
    out, lse = attention.attention(q, k, v, pat, scale)
    for i in range(N):
        r_i, c_i = divmod(i, 4)
        w, acc, total = [], [0.0] * d, 0.0
        for j in range(N):
            r_j, c_j = divmod(j, 4)
            if abs(r_i - r_j) <= 1 and abs(c_i - c_j) <= 1:
                w.append((j, scale * sum(q[0, 0, i, t] * k[0, 0, j, t] for t in range(d))))
        m = max(s for _, s in w)
        for j, s in w:
            e = math.exp(s - m)
            total += e
            for t in range(d):
                acc[t] += e * v[0, 0, j, t]
        for t in range(d):
            assert abs(out[0, 0, i, t] - acc[t] / total) < 1e-12
        assert abs(lse[0, 0, i] - (m + math.log(total))) < 1e-12


@pytest.mark.parametrize("pat", [Pat("hilbert_window", 8, 8, 64), Pat("hilbert_slide", 8, 8, 63),
                                 Pat("hilbert_window", 8, 8, 1000)], ids=repr)
def test_all_allowed_is_plain_attention(pat):
    N, d = 64, 16
    q, k, v = (rand((1, 2, N, d), s) for s in (7, 8, 9))
    out, lse = attention.attention(q, k, v, pat, 0.25)
    qt, kt, vt = (torch.from_numpy(a) for a in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=0.25).numpy()
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    ref_lse = torch.logsumexp(0.25 * (qt @ kt.transpose(-1, -2)), dim=-1).numpy()
    np.testing.assert_allclose(lse, ref_lse, rtol=0, atol=1e-12)


@pytest.mark.parametrize("pat", [Pat("hilbert_window", 8, 8, 1), Pat("hilbert_slide", 8, 8, 0),
                                 Pat("rowmajor_slide", 8, 8, 0, 0),
                                 Pat("rowmajor_window", 8, 8, 1, 1)], ids=repr)
def test_diagonal_mask_returns_v(pat):
    N, d = 64, 8
    q, k, v = (rand((2, 1, N, d), s) for s in (10, 11, 12))
    out, lse = attention.attention(q, k, v, pat, 0.5)
    np.testing.assert_array_equal(out, v)
    np.testing.assert_allclose(lse, 0.5 * np.einsum("bhnd,bhnd->bhn", q, k), rtol=0, atol=1e-14)


def test_rows_subset_and_softmax_weights_sum_to_one():
    pat = Pat("hilbert_slide", 16, 16, 20)
    N, d = 256, 16
    q, k, v = (rand((1, 2, N, d), s) for s in (13, 14, 15))
    full_out, full_lse = attention.attention(q, k, v, pat, 0.3)
    rows = np.array([0, 5, 100, 255, 17])
    out, lse = attention.attention(q, k, v, pat, 0.3, rows=rows)
    np.testing.assert_array_equal(out, full_out[:, :, rows])
    np.testing.assert_array_equal(lse, full_lse[:, :, rows])
    # with v = 1 the output is the row sum of the softmax weights
    ones = np.ones((1, 2, N, 3))
    o1, _ = attention.attention(q, k, ones, pat, 0.3)
    np.testing.assert_allclose(o1, 1.0, rtol=0, atol=1e-14)


@pytest.mark.parametrize("kind,p0", [("hilbert_window", 64), ("hilbert_slide", 40),
                                     ("hilbert_neighborhood", 81)])
def test_gather_attend_scatter_equals_rowmajor_with_hilbert_positions(kind, p0):
    H = W = 16
    N, d = H * W, 8
    order = hilbert.hilbert_order(H, W)
    rank = hilbert.inverse_permutation(order)
    q, k, v = (rand((1, 2, N, d), s) for s in (16, 17, 18))
    pat = Pat(kind, H, W, p0)
    oh, lh = attention.attention(permute.gather(q, order), permute.gather(k, order),
                                 permute.gather(v, order), pat, 0.35)
    orm, lrm = attention.attention(q, k, v, pat, 0.35, positions=rank)
    np.testing.assert_allclose(permute.scatter(oh, order), orm, rtol=0, atol=1e-13)
    np.testing.assert_allclose(permute.scatter(lh[..., None], order)[..., 0], lrm, rtol=0, atol=1e-13)


def test_gather_scatter_roundtrip_and_identity():
    x = rand((2, 3, 64, 5), 19)
    order = hilbert.hilbert_order(8, 8)
    assert np.array_equal(permute.scatter(permute.gather(x, order), order), x)
    assert np.array_equal(permute.gather(x, np.arange(64)), x)
    assert np.array_equal(permute.gather(x, order)[..., 3, :], x[..., order[3], :])


def test_layer_identity_weights_is_plain_attention():
    H = W = 8
    N, heads, d = 64, 2, 4
    C = heads * d
    x = rand((2, N, C), 20)
    eye = np.eye(C)
    y = layer.hnt_layer(x, np.concatenate([eye, eye, eye]), eye, H, W, heads, 5, 0.5)
    xh = x.reshape(2, N, heads, d).transpose(0, 2, 1, 3)
    rank = hilbert.hilbert_rank(H, W)
    o, _ = attention.attention(xh, xh, xh, Pat("hilbert_slide", H, W, 5), 0.5, positions=rank)
    np.testing.assert_allclose(y, o.transpose(0, 2, 1, 3).reshape(2, N, C), rtol=0, atol=1e-13)


def test_layer_equals_hilbert_order_pipeline():
    """Row-major formulation == gather -> project -> Hilbert slide -> project -> scatter."""
    H = W = 16
    N, heads, d, h = 256, 3, 8, 12
    C = heads * d
    x = rand((2, N, C), 21)
    wq = rand((3 * C, C), 22, 0.1)
    wp = rand((C, C), 23, 0.1)
    y = layer.hnt_layer(x, wq, wp, H, W, heads, h, 0.3)
    order = hilbert.hilbert_order(H, W)
    xh = permute.gather(x, order)
    qkv = (xh @ wq.T).reshape(2, N, 3, heads, d).transpose(2, 0, 3, 1, 4)
    o, _ = attention.attention(qkv[0], qkv[1], qkv[2], Pat("hilbert_slide", H, W, h), 0.3)
    yh = o.transpose(0, 2, 1, 3).reshape(2, N, C) @ wp.T
    np.testing.assert_allclose(y, permute.scatter(yh, order), rtol=0, atol=1e-12)
    rows = np.array([3, 77, 200])
    np.testing.assert_allclose(layer.hnt_layer(x, wq, wp, H, W, heads, h, 0.3, rows=rows),
                               y[:, rows], rtol=0, atol=1e-13)
