"""Pins for the oracle's Hilbert order (recursive quadrant construction).

The paper names the Hilbert curve for its locality (Sec. 1, Sec. 3.1) and caches
one path per feature-map size (Sec. 3.2); it fixes no orientation. These tests
pin the oracle to what any Hilbert curve must satisfy, and to the textbook
iterative index-to-cell algorithm and its inverse (the quadrant-rotation loop of Hacker's
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


def textbook_xy2d(side, x, y):
    """Iterative (x, y) -> d on a side x side curve, the inverse of textbook_d2xy:
    per level from the coarsest, read the quadrant bits, add its offset, then
    undo the rotation/reflection of the low bits."""
    d = 0
    s = side // 2
    while s > 0:
        rx = 1 if x & s else 0
        ry = 1 if y & s else 0
        d += s * s * ((3 * rx) ^ ry)
        if ry == 0:
            if rx == 1:
                x, y = s - 1 - (x & (s - 1)), s - 1 - (y & (s - 1))
            x, y = y, x
        s //= 2
    return d


def test_textbook_pair_are_inverses():
    for side in (1, 2, 4, 8, 16):
        for d in range(side * side):
            x, y = textbook_d2xy(side, d)
            assert textbook_xy2d(side, x, y) == d


GRIDS = [(1, 1), (1, 7), (7, 1), (3, 5), (5, 3), (6, 6), (7, 13), (17, 9), (24, 24), (32, 48),
         (48, 32), (56, 56), (64, 128), (128, 64), (96, 96), (100, 37), (160, 160), (128, 256)]


@pytest.mark.parametrize("H,W", GRIDS)
def test_any_grid_is_a_bijection(H, W):
    order = hilbert.hilbert_order(H, W)
    assert order.shape == (H * W,)
    assert np.array_equal(np.sort(order), np.arange(H * W))


@pytest.mark.parametrize("H,W", GRIDS)
def test_any_grid_follows_the_enclosing_curve(H, W):
    """Every cell of the grid appears, and their positions on the enclosing
    2^k curve (computed with the textbook inverse, not the oracle) increase."""
    side = 1
    while side < max(H, W):
        side *= 2
    order = hilbert.hilbert_order(H, W)
    pos = [textbook_xy2d(side, int(t) % W, int(t) // W) for t in order]
    assert all(a < b for a, b in zip(pos, pos[1:]))
    assert len(pos) == H * W


@pytest.mark.parametrize("k", range(1, 8))
def test_two_to_one_rectangles(k):
    """A 2^k x 2^(k+1) grid (rows x cols) is the lower half of the enclosing square:
    the path is one 2^k square curve after the other, with a single jump between
    them; a 2^(k+1) x 2^k grid is the left half and the path never jumps."""
    s = 1 << k
    wide = hilbert.hilbert_order(s, 2 * s)
    x, y = wide % (2 * s), wide // (2 * s)
    assert (x[: s * s] < s).all() and (x[s * s:] >= s).all()
    steps = np.abs(np.diff(x)) + np.abs(np.diff(y))
    assert (steps != 1).sum() == 1 and steps[s * s - 1] != 1
    tall = hilbert.hilbert_order(2 * s, s)
    x, y = tall % s, tall // s
    assert (np.abs(np.diff(x)) + np.abs(np.diff(y)) == 1).all()


def test_rejects_empty_grid():
    with pytest.raises(ValueError):
        hilbert.hilbert_order(0, 4)
