"""Pins for the oracle's Hilbert order (recursive quadrant construction).

The paper names the Hilbert curve for its locality (Sec. 1, Sec. 3.1) and caches
one path per feature-map size (Sec. 3.2); it fixes no orientation. These tests
pin the oracle to what any Hilbert curve must satisfy, and to the textbook
iterative index-to-cell algorithm (the quadrant-rotation loop of Hacker's
Delight, ch. 16, also given on Wikipedia's "Hilbert curve" page), written out
here independently of the oracle's recursion.
"""
import numpy as np
import pytest

from oracle import hilbert


def textbook_d2xy(side, d):
    """Iterative d -> (x, y): per level, pick the quadrant from two bits of d,
    rotate/reflect the partial point, then offset it into the quadrant."""
    x = y = 0
    s = 1
    t = d
    while s < side:
        rx = 1 & (t // 2)
        ry = 1 & (t ^ rx)
        if ry == 0:
            if rx == 1:
                x, y = s - 1 - x, s - 1 - y
            x, y = y, x
        x += s * rx
        y += s * ry
        t //= 4
        s *= 2
    return x, y


@pytest.mark.parametrize("k", range(0, 11))
def test_bijection(k):
    side = 1 << k
    order = hilbert.hilbert_order(side, side)
    assert order.shape == (side * side,)
    assert np.array_equal(np.sort(order), np.arange(side * side))
    rank = hilbert.inverse_permutation(order)
    assert np.array_equal(order[rank], np.arange(side * side))
    assert np.array_equal(rank[order], np.arange(side * side))


@pytest.mark.parametrize("k", range(1, 11))
def test_consecutive_cells_are_4_adjacent(k):
    cells = hilbert.hilbert_cells(k)
    step = np.abs(np.diff(cells, axis=0)).sum(axis=1)
    assert (step == 1).all()


@pytest.mark.parametrize("k", range(0, 13))
def test_matches_textbook_iterative(k):
    side = 1 << k
    cells = hilbert.hilbert_cells(k)
    if side * side > 1 << 16:
        idx = np.random.default_rng(k).choice(side * side, 4096, replace=False)
    else:
        idx = np.arange(side * side)
    for d in idx:
        assert tuple(cells[d]) == textbook_d2xy(side, int(d)), (k, d)


@pytest.mark.parametrize("k", range(1, 9))
def test_power_of_four_windows_are_aligned_squares(k):
    """Every Hilbert window of 4^m consecutive positions covers one aligned 2^m x 2^m block."""
    cells = hilbert.hilbert_cells(k)
    for m in range(0, k + 1):
        w = 4 ** m
        s = 1 << m
        blocks = cells.reshape(-1, w, 2)
        x0 = blocks[:, :, 0].min(axis=1)
        y0 = blocks[:, :, 1].min(axis=1)
        assert (x0 % s == 0).all() and (y0 % s == 0).all()
        assert (blocks[:, :, 0].max(axis=1) - x0 == s - 1).all()
        assert (blocks[:, :, 1].max(axis=1) - y0 == s - 1).all()
        # all w cells distinct inside the s x s square
        ids = (blocks[:, :, 1] - y0[:, None]) * s + (blocks[:, :, 0] - x0[:, None])
        assert (np.sort(ids, axis=1) == np.arange(w)).all()


@pytest.mark.parametrize("k", range(1, 9))
def test_endpoints(k):
    cells = hilbert.hilbert_cells(k)
    side = 1 << k
    assert tuple(cells[0]) == (0, 0)
    assert tuple(cells[-1]) == (side - 1, 0)


def test_small_orders_by_hand():
    # Order 1: (0,0) -> up to (0,1) -> right to (1,1) -> down to (1,0).
    assert hilbert.hilbert_order(2, 2).tolist() == [0, 2, 3, 1]
    # Order 2, traced from the same convention on a 4x4 grid (id = 4*y + x).
    assert hilbert.hilbert_order(4, 4).tolist() == [0, 1, 5, 4, 8, 12, 13, 9,
                                                   10, 14, 15, 11, 7, 6, 2, 3]


def test_rejects_non_power_of_two():
    with pytest.raises(ValueError):
        hilbert.hilbert_order(96, 96)
    with pytest.raises(ValueError):
        hilbert.hilbert_order(64, 128)
