"""Pins for the oracle's element masks and brute-force tile classifier.

Pinned to the block counts the paper prints: the Fig. 3 worked example (Sec. 3.1)
and the empty-tile percentages of Tables 1-3, 6, 9 and 11. Also to closed forms
(Hilbert window: N/w diagonal groups of full tiles), to the band's interval
bounds, and to brute force on tiny grids.
"""
import numpy as np
import pytest

from conftest import Pat, read_golden
from oracle import blockmask, masks

SPARSITY = read_golden("paper_sparsity.txt")
FIG3 = read_golden("fig3_example.txt")


@pytest.mark.parametrize("row", SPARSITY, ids=[s for _, s in SPARSITY])
def test_paper_sparsity(row):
    (kind, H, W, p0, p1, block, printed), source = row
    pat = Pat(kind, H, W, p0, p1)
    b = int(block)
    pct = 100.0 * blockmask.block_sparsity(pat, b)
    assert round(pct, 2) == pytest.approx(float(printed), abs=1e-9), (source, pct)
    if (pat.H * pat.W) % b == 0:   # whole tiles: the same number as the share of empty tiles
        assert pct == pytest.approx(100.0 * blockmask.empty_fraction(pat, b, b), abs=1e-9)


@pytest.mark.parametrize("row", FIG3, ids=[s for _, s in FIG3])
def test_fig3_worked_example(row):
    (kind, H, W, p0, p1, block, full, part, empty), source = row
    pat = Pat(kind, H, W, p0, p1)
    b = int(block)
    cls = blockmask.classify(pat, b, b)[:2, :2]     # first eight tokens
    assert int((cls == blockmask.FULL).sum()) == int(full), source
    assert int((cls == blockmask.PARTIAL).sum()) == int(part), source
    assert int((cls == blockmask.EMPTY).sum()) == int(empty), source


def test_fig3_wsa_partials_are_half_full():
    pat = Pat("rowmajor_window", 4, 4, 2, 2)
    counts = blockmask.tile_counts(pat, 4, 4)[:2, :2]
    assert (counts == 8).all()   # 8 of 16 elements: half full


def test_fig3_windows_follow_token_lists():
    # Row-major 2x2 windows: first window tokens (1,2,5,6), second (3,4,7,8), 1-based.
    m = masks.dense(Pat("rowmajor_window", 4, 4, 2, 2))
    assert sorted(np.nonzero(m[0])[0] + 1) == [1, 2, 5, 6]
    assert sorted(np.nonzero(m[2])[0] + 1) == [3, 4, 7, 8]
    # Hilbert windows: (1,2,3,4) and (5,6,7,8).
    mh = masks.dense(Pat("hilbert_window", 4, 4, 4))
    assert sorted(np.nonzero(mh[0])[0] + 1) == [1, 2, 3, 4]
    assert sorted(np.nonzero(mh[4])[0] + 1) == [5, 6, 7, 8]


@pytest.mark.parametrize("N,w,bm,bn", [(1024, 64, 64, 64), (16384, 256, 128, 64),
                                       (4096, 256, 128, 128), (4096, 1024, 128, 64),
                                       (4096, 128, 128, 64)])
def test_hilbert_window_diagonal_groups(N, w, bm, bn):
    """With both tile sizes dividing w: exactly N/w groups of (w/bm)(w/bn) full tiles on the
    diagonal, no partial tile."""
    side = int(round(N ** 0.5))
    bmk = blockmask.build(Pat("hilbert_window", side, side, w), bm, bn)
    assert bmk.total_part == 0
    assert bmk.total_full == (N // w) * (w // bm) * (w // bn)
    # the full tiles form N/w diagonal groups: tile (qt, kt) full iff same window group
    qt = np.arange(N // bm)[:, None]
    kt = np.arange(N // bn)[None, :]
    assert np.array_equal(bmk.cls == blockmask.FULL, (qt * bm) // w == (kt * bn) // w)


@pytest.mark.parametrize("N,h,bm,bn", [(4096, 128, 128, 64), (1024, 40, 64, 64),
                                       (1024, 0, 64, 32), (1024, 1023, 64, 64),
                                       (4096, 64, 128, 64), (4096, 512, 128, 128)])
def test_band_interval_bounds(N, h, bm, bn):
    """Band |i-j| <= h: a tile is empty iff its closest pair is farther than h, full iff its
    farthest pair is within h (the tile's index ranges are intervals)."""
    side = int(round(N ** 0.5))
    cls = blockmask.classify(Pat("hilbert_slide", side, side, h), bm, bn)
    for qt in range(N // bm):
        i0, i1 = qt * bm, qt * bm + bm - 1
        for kt in range(N // bn):
            j0, j1 = kt * bn, kt * bn + bn - 1
            dmin = max(0, j0 - i1, i0 - j1)
            dmax = max(abs(i0 - j1), abs(i1 - j0))
            want = blockmask.EMPTY if dmin > h else (blockmask.FULL if dmax <= h else blockmask.PARTIAL)
            assert cls[qt, kt] == want


def test_band_counts_for_the_slide_workload():
    # 64x64 grid, band +-128, tiles 128x64: 64 full + 124 partial non-empty tiles.
    bmk = blockmask.build(Pat("hilbert_slide", 64, 64, 128), 128, 64)
    assert (bmk.total_full, bmk.total_part) == (64, 124)


def brute_force_tiny(pat, bm, bn):
    """Literal element-by-element loop (tiny grids only). Slots past N (ragged edge
    tiles) are never allowed."""
    N = pat.H * pat.W
    m = masks.dense(pat)
    nq, nk = (N + bm - 1) // bm, (N + bn - 1) // bn
    cls = np.zeros((nq, nk), dtype=np.int8)
    for qt in range(nq):
        for kt in range(nk):
            c = 0
            for i in range(qt * bm, qt * bm + bm):
                for j in range(kt * bn, kt * bn + bn):
                    if i < N and j < N:
                        c += int(m[i, j])
            cls[qt, kt] = 0 if c == 0 else (2 if c == bm * bn else 1)
    return cls


@pytest.mark.parametrize("pat,bm,bn", [
    (Pat("rowmajor_window", 8, 8, 2, 4), 8, 4),
    (Pat("rowmajor_slide", 8, 8, 1, 2), 4, 8),
    (Pat("hilbert_window", 8, 8, 8), 4, 4),
    (Pat("hilbert_slide", 8, 8, 5), 8, 8),
    (Pat("hilbert_neighborhood", 8, 8, 9), 4, 8),
    (Pat("rowmajor_neighborhood", 8, 8, 3, 3), 8, 4),
    (Pat("hilbert_shifted_window", 8, 8, 8, 4), 4, 4),
])
def test_classifier_matches_literal_loop(pat, bm, bn):
    assert np.array_equal(blockmask.classify(pat, bm, bn), brute_force_tiny(pat, bm, bn))


@pytest.mark.parametrize("pat,bm,bn", [
    (Pat("rowmajor_window", 7, 7, 3, 2), 8, 4),
    (Pat("rowmajor_slide", 5, 9, 1, 2), 16, 8),
    (Pat("hilbert_window", 7, 7, 8), 4, 16),
    (Pat("hilbert_slide", 6, 5, 3), 8, 8),
    (Pat("hilbert_neighborhood", 7, 6, 9), 16, 4),
    (Pat("rowmajor_neighborhood", 7, 7, 3, 3), 8, 16),
    (Pat("hilbert_shifted_window", 9, 7, 8, 3), 8, 8),
])
def test_ragged_classifier_matches_literal_loop(pat, bm, bn):
    """N not a multiple of the tiles: ceil(N / b) tiles per axis, padded slots never allowed."""
    cls = blockmask.classify(pat, bm, bn)
    assert np.array_equal(cls, brute_force_tiny(pat, bm, bn))
    N = pat.H * pat.W
    assert cls.shape == ((N + bm - 1) // bm, (N + bn - 1) // bn)
    if N % bn:
        assert (cls[:, -1] != blockmask.FULL).all()     # an edge tile is never full
    if N % bm:
        assert (cls[-1, :] != blockmask.FULL).all()


@pytest.mark.parametrize("H,W,h,bm,bn", [(56, 56, 24, 128, 64), (56, 56, 512, 128, 128),
                                         (10, 10, 7, 64, 16), (7, 9, 0, 16, 32)])
def test_ragged_band_interval_bounds(H, W, h, bm, bn):
    """Band on a ragged tiling: the tile's real index ranges are intervals clipped at N - 1;
    empty iff their closest pair is farther than h, full iff the tile is whole and its
    farthest pair is within h."""
    N = H * W
    cls = blockmask.classify(Pat("hilbert_slide", H, W, h), bm, bn)
    for qt in range((N + bm - 1) // bm):
        i0, i1 = qt * bm, min(N, qt * bm + bm) - 1
        for kt in range((N + bn - 1) // bn):
            j0, j1 = kt * bn, min(N, kt * bn + bn) - 1
            whole = i1 - i0 + 1 == bm and j1 - j0 + 1 == bn
            dmin = max(0, j0 - i1, i0 - j1)
            dmax = max(abs(i0 - j1), abs(i1 - j0))
            want = (blockmask.EMPTY if dmin > h else
                    blockmask.FULL if whole and dmax <= h else blockmask.PARTIAL)
            assert cls[qt, kt] == want


def test_lists_are_ascending_and_padded():
    bmk = blockmask.build(Pat("rowmajor_slide", 16, 16, 2, 2), 32, 16)
    nq, nk = bmk.cls.shape
    for q in range(nq):
        f = bmk.full_idx[q, :bmk.n_full[q]]
        p = bmk.part_idx[q, :bmk.n_part[q]]
        assert (np.diff(f) > 0).all() and (np.diff(p) > 0).all()
        assert (bmk.full_idx[q, bmk.n_full[q]:] == -1).all()
        assert (bmk.part_idx[q, bmk.n_part[q]:] == -1).all()
        assert set(f) == set(np.nonzero(bmk.cls[q] == blockmask.FULL)[0])
        assert set(p) == set(np.nonzero(bmk.cls[q] == blockmask.PARTIAL)[0])


def test_every_query_attends_itself():
    for pat in [Pat("hilbert_window", 16, 16, 16), Pat("hilbert_slide", 16, 16, 0),
                Pat("rowmajor_window", 16, 16, 4, 4), Pat("rowmajor_slide", 16, 16, 0, 0),
                Pat("hilbert_neighborhood", 16, 16, 9), Pat("rowmajor_neighborhood", 16, 16, 3, 3),
                Pat("hilbert_shifted_window", 16, 16, 16, 8)]:
        assert np.diag(masks.dense(pat)).all(), pat


def test_neighborhood_has_constant_size_and_slide_truncates():
    N = 256
    nh = masks.dense(Pat("hilbert_neighborhood", 16, 16, 9))
    assert (nh.sum(axis=1) == 9).all()             # clamped windows keep k keys
    sl = masks.dense(Pat("hilbert_slide", 16, 16, 4))
    assert sl[0].sum() == 5 and sl[N // 2].sum() == 9   # band truncates at the ends
    na = masks.dense(Pat("rowmajor_neighborhood", 16, 16, 3, 3))
    assert (na.sum(axis=1) == 9).all()


def test_shifted_window_masks_the_wrapped_pair():
    # w = 16, s = 8 on 256 positions: windows [0,8), [8,24), ..., [248,256); the head and the
    # tail (which a cyclic roll would put in one window) never attend each other.
    m = masks.dense(Pat("hilbert_shifted_window", 16, 16, 16, 8))
    assert not m[0, 255] and not m[255, 0]
    assert m[8, 23] and not m[7, 8]
    assert m[:8, :8].all() and m[248:, 248:].all()


def test_shifted_window_moves_each_window_forward():
    """Sec. 3.2: the shifted windows are the plain windows moved forward along the
    sequence by s. With w = 16 and s = 4 on 256 positions the windows are [0, 4),
    [4, 20), [20, 36), ..., [244, 256). A shift that moved them the other way
    (window id floor((i + s) / w), the same as this one only at s = w / 2) would
    give [0, 12), [12, 28), ... instead, and fails every check below."""
    m = masks.dense(Pat("hilbert_shifted_window", 16, 16, 16, 4))
    assert m[:4, :4].all() and not m[3, 4] and not m[4, 3]
    assert m[4:20, 4:20].all() and not m[19, 20] and not m[20, 19]
    assert m[4, 11] and m[11, 12]                  # [0, 12) / [12, 28) would split these
    assert m[244:, 244:].all() and not m[243, 244]
    assert not m[0, 255] and not m[255, 0]
    sizes = m.sum(axis=1)
    assert (sizes[:4] == 4).all() and (sizes[4:244] == 16).all() and (sizes[244:] == 12).all()


def _swin_shifted_mask(N, w, s):
    """The shifted-window mask built the way the Swin Transformer builds it, on a 1-D
    sequence (the construction Sec. 3.2 moves onto the Hilbert sequence): roll the
    sequence back by s (rolled position t holds token (t + s) mod N), cut the rolled
    sequence into windows of w, label the regions [0, N - w), [N - w, N - s),
    [N - s, N) of the rolled sequence, and allow a pair when it shares a window and a
    label (the label masks the pairs the roll joined across the sequence ends)."""
    t = (np.arange(N) - s) % N                       # rolled position of each token
    label = np.where(t < N - w, 0, np.where(t < N - s, 1, 2))
    win = t // w
    return (win[:, None] == win[None, :]) & (label[:, None] == label[None, :])


@pytest.mark.parametrize("H,W,w,s", [(16, 16, 16, 4), (16, 16, 16, 13), (16, 16, 64, 5),
                                     (8, 8, 8, 1), (16, 16, 16, 8), (32, 32, 64, 48)])
def test_shifted_window_equals_the_swin_roll_construction(H, W, w, s):
    m = masks.dense(Pat("hilbert_shifted_window", H, W, w, s))
    assert np.array_equal(m, _swin_shifted_mask(H * W, w, s))
