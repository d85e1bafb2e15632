"""Pins for the oracle's attention gradients and the per-column tile lists.

The gradients are pinned to things other than their own formulas:
  - PyTorch autograd (float64, CPU) through a directly written masked softmax
    attention: a differentiation the oracle does not perform;
  - central finite differences of the scalar <dout, out> on tiny inputs;
  - closed forms: a diagonal-only mask gives out = v, so dv = dout and dq = dk = 0;
  - invariances of the forward that fix sums of the gradients exactly: adding a
    vector to every key leaves every softmax row unchanged (sum_j dk_j = 0);
    adding a vector to every value adds it to every output (sum_j dv_j =
    sum_i dout_i); scaling q by t and k by 1/t leaves the scores unchanged
    (sum_i <dq_i, q_i> = sum_j <dk_j, k_j>);
  - restricting the outputs to subsets of rows and keys equals slicing the full
    result, and Hilbert attention on gathered tensors equals the same pattern on
    Hilbert positions of row-major tensors (gradients gathered alike).
"""
import math

import numpy as np
import pytest
import torch

from conftest import Pat
from oracle import attention, blockmask, hilbert, masks


def rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def autograd_ref(q, k, v, dout, mask, scale):
    qt, kt, vt = (torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (q, k, v))
    s = (qt @ kt.transpose(-1, -2)) * scale
    s = s.masked_fill(~torch.from_numpy(mask), float("-inf"))
    p = torch.softmax(s, dim=-1)
    out = p @ vt
    out.backward(torch.from_numpy(dout))
    return qt.grad.numpy(), kt.grad.numpy(), vt.grad.numpy()


PATS = [Pat("hilbert_window", 8, 8, 16), Pat("hilbert_slide", 8, 8, 6),
        Pat("rowmajor_window", 8, 8, 2, 4), Pat("rowmajor_slide", 8, 8, 1, 2),
        Pat("hilbert_neighborhood", 8, 8, 9), Pat("rowmajor_neighborhood", 8, 8, 3, 5),
        Pat("hilbert_shifted_window", 8, 8, 16, 8), Pat("hilbert_slide", 16, 16, 40)]


@pytest.mark.parametrize("pat", PATS, ids=repr)
@pytest.mark.parametrize("d", [4, 32])
def test_matches_autograd(pat, d):
    N = pat.N
    q, k, v, do = (rand((2, 2, N, d), s) for s in (11, 12, 13, 14))
    scale = 1 / math.sqrt(d)
    got = attention.attention_backward(q, k, v, do, pat, scale, chunk=29)
    ref = autograd_ref(q, k, v, do, masks.dense(pat), scale)
    for g, r, name in zip(got, ref, ("dq", "dk", "dv")):
        np.testing.assert_allclose(g, r, rtol=0, atol=1e-12, err_msg=name)


def test_finite_differences():
    pat = Pat("hilbert_neighborhood", 4, 4, 5)
    N, d, scale = 16, 3, 0.7
    q, k, v, do = (rand((1, 1, N, d), s) for s in (21, 22, 23, 24))

    def loss(q_, k_, v_):
        out, _ = attention.attention(q_, k_, v_, pat, scale)
        return float((out * do).sum())

    dq, dk, dv = attention.attention_backward(q, k, v, do, pat, scale)
    eps = 1e-6
    for which, grad in ((0, dq), (1, dk), (2, dv)):
        for seed in range(3):
            u = rand(q.shape, 100 + 10 * which + seed)
            args_p = [q, k, v]
            args_m = [q, k, v]
            args_p[which] = args_p[which] + eps * u
            args_m[which] = args_m[which] - eps * u
            fd = (loss(*args_p) - loss(*args_m)) / (2 * eps)
            assert abs(fd - float((grad * u).sum())) < 1e-7, (which, seed)


def test_diagonal_mask_closed_form():
    pat = Pat("hilbert_window", 8, 8, 1)
    q, k, v, do = (rand((2, 3, 64, 16), s) for s in (31, 32, 33, 34))
    dq, dk, dv = attention.attention_backward(q, k, v, do, pat, 0.25)
    assert np.array_equal(dv, do)
    assert not dq.any() and not dk.any()


@pytest.mark.parametrize("pat", PATS[:7], ids=repr)
def test_invariance_sums(pat):
    N, d = pat.N, 8
    q, k, v, do = (rand((1, 2, N, d), s) for s in (41, 42, 43, 44))
    dq, dk, dv = attention.attention_backward(q, k, v, do, pat, 0.3)
    np.testing.assert_allclose(dk.sum(axis=2), 0.0, atol=1e-12)
    np.testing.assert_allclose(dv.sum(axis=2), do.sum(axis=2), atol=1e-12)
    np.testing.assert_allclose((dq * q).sum(axis=(2, 3)), (dk * k).sum(axis=(2, 3)), atol=1e-12)


def test_restricted_rows_and_keys_equal_slices():
    pat = Pat("hilbert_slide", 16, 16, 21)
    q, k, v, do = (rand((2, 2, 256, 8), s) for s in (51, 52, 53, 54))
    full = attention.attention_backward(q, k, v, do, pat, 0.35)
    rows = np.array([0, 5, 77, 128, 255])
    keys = np.array([3, 100, 101, 250])
    dq, dk, dv = attention.attention_backward(q, k, v, do, pat, 0.35, rows=rows, key_rows=keys,
                                              chunk=17)
    np.testing.assert_allclose(dq, full[0][:, :, rows], rtol=0, atol=1e-13)
    np.testing.assert_allclose(dk, full[1][:, :, keys], rtol=0, atol=1e-13)
    np.testing.assert_allclose(dv, full[2][:, :, keys], rtol=0, atol=1e-13)


def test_hilbert_equivariance():
    pat = Pat("hilbert_slide", 8, 8, 7)
    order = hilbert.hilbert_order(8, 8)
    rank = hilbert.inverse_permutation(order)
    q, k, v, do = (rand((1, 2, 64, 8), s) for s in (61, 62, 63, 64))
    g_row = attention.attention_backward(q, k, v, do, pat, 0.4, positions=rank)
    g_hil = attention.attention_backward(q[:, :, order], k[:, :, order], v[:, :, order],
                                         do[:, :, order], pat, 0.4)
    for a, b in zip(g_row, g_hil):
        np.testing.assert_allclose(a[:, :, order], b, rtol=0, atol=1e-12)


@pytest.mark.parametrize("pat", PATS[:7], ids=repr)
def test_column_lists_cover_the_transposed_mask(pat):
    """Column lists hold exactly the query tiles whose tile with the key tile is
    full / partial, ascending: checked against the element mask directly."""
    tm, tn = 16, 8
    cls = blockmask.classify(pat, tm, tn)
    cols = blockmask.column_lists(cls)
    dense = masks.dense(pat)
    nq, nk = pat.N // tm, pat.N // tn
    for kt in range(nk):
        full, part = [], []
        for qt in range(nq):
            c = int(dense[qt * tm:(qt + 1) * tm, kt * tn:(kt + 1) * tn].sum())
            if c == tm * tn:
                full.append(qt)
            elif c:
                part.append(qt)
        assert cols.n_full[kt] == len(full) and cols.n_part[kt] == len(part)
        assert list(cols.full_idx[kt, :len(full)]) == full
        assert list(cols.part_idx[kt, :len(part)]) == part
        assert (cols.full_idx[kt, len(full):] == -1).all()
        assert (cols.part_idx[kt, len(part):] == -1).all()
