"""GPU parity: tile classes and lists are bit-exact against the brute-force oracle
(every query-tile row of every measured workload), and the empty-tile fractions
equal the values the paper prints."""
import numpy as np
import pytest

import oracle_pool
import paper_2511_05832_amd as hla
import workloads as W
from conftest import Pat, read_golden
from helpers import assert_mask_matches_oracle, gpu_block_mask_host

pytestmark = pytest.mark.gpu

ATTN = [w for w in W.ATTN_WORKLOADS] + [W.C5]


@pytest.mark.parametrize("w", ATTN, ids=lambda w: w.name)
def test_workload_masks_bit_exact(w):
    """Every query-tile row (512 on the 256 x 256 grid) against the brute-force oracle;
    the large grids' rows are evaluated in chunks across worker processes."""
    pat = w.pattern
    mask = hla.build_block_mask(pat, w.tile_m, w.tile_n)
    nq = mask.n_qtiles
    if nq <= 128:
        assert_mask_matches_oracle(mask, pat, w.tile_m, w.tile_n)
    else:
        got = gpu_block_mask_host(mask)
        ref = oracle_pool.tile_lists(pat, w.tile_m, w.tile_n, range(nq))
        for g, r, name in zip(got, ref, ("n_full", "full_idx", "n_part", "part_idx")):
            np.testing.assert_array_equal(g, r, err_msg=name)
    tf, tp = mask.host_totals()
    assert tf == int(mask.n_full.sum()) and tp == int(mask.n_part.sum())


# full and partial tiles per (b, h), from the oracle over every row
TILE_COUNTS = {r[0][0]: (int(r[0][3]), int(r[0][4])) for r in read_golden("tile_counts.txt")}


@pytest.mark.parametrize("w", ATTN, ids=lambda w: w.name)
def test_workload_tile_counts(w):
    mask = hla.build_block_mask(w.pattern, w.tile_m, w.tile_n)
    assert mask.host_totals() == TILE_COUNTS[w.name]


@pytest.mark.parametrize("row", read_golden("paper_sparsity.txt"), ids=lambda r: r[1])
def test_paper_sparsity_on_gpu(row):
    (kind, H, Wd, p0, p1, block, printed), source = row
    b = int(block)
    pat = Pat(kind, H, Wd, p0, p1)
    mask = hla.build_block_mask(pat, b, b)
    tf, tp = mask.host_totals()
    # share of the score matrix outside the non-empty b x b blocks (the share of
    # empty tiles when b divides N; ragged 56 x 56 rows count whole blocks)
    pct = 100.0 * (1.0 - (tf + tp) * b * b / float(pat.N) ** 2)
    assert round(pct, 2) == pytest.approx(float(printed), abs=1e-9), source


def random_patterns(n):
    rng = np.random.default_rng(1234)
    out = []
    kinds = list(hla.PATTERN_IDS)
    for i in range(n):
        kind = kinds[i % len(kinds)]
        H = int(rng.choice([8, 12, 16, 24, 32]))
        Wd = int(rng.choice([8, 16, 20, 32, 48]))
        N = H * Wd
        if kind == "hilbert_window":
            pat = Pat(kind, H, Wd, int(rng.integers(1, N + 40)))
        elif kind == "hilbert_slide":
            pat = Pat(kind, H, Wd, int(rng.integers(0, N)))
        elif kind == "hilbert_neighborhood":
            pat = Pat(kind, H, Wd, int(rng.integers(1, N + 1)))
        elif kind == "hilbert_shifted_window":
            w = int(rng.integers(1, 200))
            pat = Pat(kind, H, Wd, w, int(rng.integers(0, w)))
        elif kind == "rowmajor_window":
            pat = Pat(kind, H, Wd, int(rng.integers(1, H + 3)), int(rng.integers(1, Wd + 3)))
        elif kind == "rowmajor_slide":
            pat = Pat(kind, H, Wd, int(rng.integers(0, H)), int(rng.integers(0, Wd)))
        else:
            pat = Pat(kind, H, Wd, int(rng.integers(1, H + 1)), int(rng.integers(1, Wd + 1)))
        tiles = [t for t in (16, 32, 64, 128) if N % t == 0]
        out.append((pat, int(rng.choice(tiles)), int(rng.choice(tiles))))
    return out


@pytest.mark.parametrize("pat,tm,tn", random_patterns(70), ids=lambda x: repr(x) if isinstance(x, Pat) else str(x))
def test_random_patterns_bit_exact(pat, tm, tn):
    mask = hla.build_block_mask(pat, tm, tn)
    assert_mask_matches_oracle(mask, pat, tm, tn)


@pytest.mark.parametrize("pat,tm,tn", [(Pat("hilbert_shifted_window", 32, 32, 16, 4), 16, 16),
                                       (Pat("hilbert_shifted_window", 64, 64, 256, 64), 128, 64),
                                       (Pat("hilbert_shifted_window", 64, 64, 256, 200), 64, 64)], ids=str)
def test_shifted_windows_with_an_unequal_shift(pat, tm, tn):
    mask = hla.build_block_mask(pat, tm, tn)
    assert_mask_matches_oracle(mask, pat, tm, tn)


def test_rebuild_overwrites_previous_lists():
    m = hla.BlockMask(Pat("hilbert_slide", 32, 32, 300), 64, 64)
    m.build()
    m.struct.pat = hla.PatternDesc(hla.PATTERN_IDS["hilbert_window"], 32, 32, 64, 0)
    m.build()
    assert_mask_matches_oracle(m, Pat("hilbert_window", 32, 32, 64), 64, 64)
