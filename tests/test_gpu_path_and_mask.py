"""GPU: hla_build_path_and_mask (the Hilbert index and the tile lists in one call,
one launch on 2^k x 2^k grids) equals hla_hilbert_perm followed by
hla_build_block_mask bit for bit, on squares from 4 x 4 to 4096 x 4096, on grids
without a 2^k curve (the two launches in sequence), with and without the
transposed lists and totals, and with either output left out. (The index alone
is checked against the oracle on every 2^k square up to 4096 x 4096 in
test_gpu_permute.py.)"""
import pytest
import torch

import paper_2511_05832_amd as hla
from conftest import Pat

pytestmark = pytest.mark.gpu

LISTS = ("n_full", "full_idx", "n_part", "part_idx")
COLS = ("n_full_t", "full_idx_t", "n_part_t", "part_idx_t")


def separate(pat, tm, tn, columns):
    order, rank = hla.hilbert_perm(pat.H, pat.W)
    m = hla.BlockMask(pat, tm, tn, columns=columns).build()
    return order, rank, m


@pytest.mark.parametrize("pat,tm,tn,columns", [
    (Pat("hilbert_window", 4, 4, 4), 16, 16, False),
    (Pat("hilbert_slide", 8, 8, 5), 16, 16, True),
    (Pat("hilbert_window", 128, 128, 256), 128, 64, False),
    (Pat("hilbert_slide", 256, 256, 512), 128, 64, True),
    (Pat("rowmajor_slide", 64, 64, 4, 4), 64, 64, False),
    (Pat("hilbert_shifted_window", 32, 32, 64, 16), 64, 64, True),
    (Pat("hilbert_slide", 56, 56, 24), 64, 64, False),       # no 2^k curve: two launches
    (Pat("hilbert_window", 128, 256, 256), 128, 64, True),   # 2^k x 2^(k+1)
    (Pat("hilbert_slide", 2, 2, 1), 16, 16, False),          # side < 4: two launches
], ids=str)
def test_equals_the_separate_calls(pat, tm, tn, columns):
    o_ref, r_ref, m_ref = separate(pat, tm, tn, columns)
    order = torch.full((pat.N,), -5, dtype=torch.int32, device="cuda")
    rank = torch.full((pat.N,), -5, dtype=torch.int32, device="cuda")
    m = hla.BlockMask(pat, tm, tn, columns=columns)
    for name in LISTS:
        getattr(m, name).fill_(-9)
    m.build_with_path(order, rank)
    torch.cuda.synchronize()
    assert torch.equal(order, o_ref) and torch.equal(rank, r_ref)
    for name in LISTS + (COLS if columns else ()):
        assert torch.equal(getattr(m, name), getattr(m_ref, name)), name
    assert m.host_totals() == m_ref.host_totals()


@pytest.mark.parametrize("which", ["order", "rank", "none"])
def test_either_output_may_be_left_out(which):
    pat = Pat("hilbert_window", 64, 64, 256)
    o_ref, r_ref, m_ref = separate(pat, 128, 64, False)
    order = torch.empty(pat.N, dtype=torch.int32, device="cuda") if which == "order" else None
    rank = torch.empty(pat.N, dtype=torch.int32, device="cuda") if which == "rank" else None
    m = hla.BlockMask(pat, 128, 64).build_with_path(order, rank)
    torch.cuda.synchronize()
    if order is not None:
        assert torch.equal(order, o_ref)
    if rank is not None:
        assert torch.equal(rank, r_ref)
    for name in LISTS:
        assert torch.equal(getattr(m, name), getattr(m_ref, name)), name


def test_misaligned_outputs_take_the_scalar_stores():
    """Outputs only 4-byte aligned (the documented minimum): the same values."""
    side = 64
    o_ref, r_ref = hla.hilbert_perm(side, side)
    buf = torch.empty(2 * side * side + 8, dtype=torch.int32, device="cuda")
    order, rank = buf[1:1 + side * side], buf[2 + side * side:2 + 2 * side * side]
    hla.hilbert_perm(side, side, out=(order, rank))
    torch.cuda.synchronize()
    assert torch.equal(order, o_ref) and torch.equal(rank, r_ref)
