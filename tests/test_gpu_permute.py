"""GPU parity: Hilbert index, gather and scatter are bit-exact against the oracle."""
import numpy as np
import pytest
import torch

import paper_2511_05832_amd as hla
from oracle import hilbert as o_hil
from oracle import permute as o_perm

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("k", range(0, 13))
def test_hilbert_perm_bit_exact(k):
    side = 1 << k
    order, rank = hla.hilbert_perm(side, side)
    ref = o_hil.hilbert_order(side, side)
    np.testing.assert_array_equal(order.cpu().numpy(), ref)
    np.testing.assert_array_equal(rank.cpu().numpy(), o_hil.inverse_permutation(ref))


# Grids that are not 2^k squares: the paper's 56^2, 96^2, 160^2 and 128 x 256 feature
# maps, 2:1 rectangles both ways, single rows and columns, and odd sizes.
GRIDS = [(56, 56), (96, 96), (160, 160), (128, 256), (256, 128), (1, 1), (1, 1000), (1000, 1),
         (7, 13), (33, 65), (100, 37), (3, 5), (640, 480)]


@pytest.mark.parametrize("H,W", GRIDS)
def test_hilbert_perm_any_grid_bit_exact(H, W):
    order, rank = hla.hilbert_perm(H, W)
    ref = o_hil.hilbert_order(H, W)
    np.testing.assert_array_equal(order.cpu().numpy(), ref)
    np.testing.assert_array_equal(rank.cpu().numpy(), o_hil.inverse_permutation(ref))


def test_hilbert_perm_order_only_and_rank_only():
    ref = o_hil.hilbert_order(96, 96)
    order = torch.full((96 * 96,), -1, dtype=torch.int32, device="cuda")
    rank = torch.full((96 * 96,), -1, dtype=torch.int32, device="cuda")
    hla.lib().hla_hilbert_perm(96, 96, order.data_ptr(), None, None)
    hla.lib().hla_hilbert_perm(96, 96, None, rank.data_ptr(), None)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(order.cpu().numpy(), ref)
    np.testing.assert_array_equal(rank.cpu().numpy(), o_hil.inverse_permutation(ref))


def _bits(t: torch.Tensor) -> np.ndarray:
    t = t.cpu().contiguous()
    return t.view(torch.int16).numpy() if t.element_size() == 2 else t.view(torch.int32).numpy()


SHAPES = [
    # (B, heads, N, d, dtype, order kind)
    (2, 4, 4096, 64, torch.bfloat16, "hilbert"),      # the slide workload's q/k/v
    (1, 1, 1024, 32, torch.float32, "hilbert"),       # the fp32 window workload
    (16, 1, 4096, 192, torch.bfloat16, "hilbert"),    # layer features [B, N, C]
    (3, 2, 256, 6, torch.float32, "random"),          # 24-byte rows: 8-byte vectors
    (2, 3, 1024, 2, torch.bfloat16, "random"),        # 4-byte rows
    (1, 2, 64, 12, torch.bfloat16, "random"),         # 24-byte rows, tiny N
    (1, 1, 1, 8, torch.float32, "random"),            # N = 1
    (4, 8, 16384, 64, torch.bfloat16, "hilbert"),     # the 128x128 window workload, full size
]


@pytest.mark.parametrize("B,Hh,N,d,dtype,kind", SHAPES)
def test_gather_scatter_bit_exact(B, Hh, N, d, dtype, kind):
    g = torch.Generator().manual_seed(B * 1000 + N + d)
    x = torch.randn((B, Hh, N, d), generator=g).to(dtype)
    if kind == "hilbert":
        side = int(round(N ** 0.5))
        order_np = o_hil.hilbert_order(side, side)
        order = hla.hilbert_perm(side, side)[0]
    else:
        order_np = torch.randperm(N, generator=g).numpy()
        order = torch.from_numpy(order_np.astype(np.int32)).cuda()
    xd = x.cuda()
    xh = hla.gather(xd, order)
    ref = o_perm.gather(_bits(x), order_np)
    np.testing.assert_array_equal(_bits(xh), ref)
    back = hla.scatter(xh, order)
    np.testing.assert_array_equal(_bits(back), _bits(x))
    y = torch.randn((B, Hh, N, d), generator=g).to(dtype)
    ys = hla.scatter(y.cuda(), order)
    np.testing.assert_array_equal(_bits(ys), o_perm.scatter(_bits(y), order_np))


def test_gather_three_dim_features_and_identity():
    x = torch.randn((2, 256, 64)).to(torch.bfloat16).cuda()
    ident = torch.arange(256, dtype=torch.int32, device="cuda")
    np.testing.assert_array_equal(_bits(hla.gather(x, ident)), _bits(x))


def test_gather_rejects_wrong_order_length():
    x = torch.zeros((1, 1, 64, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(hla.HLAError):
        hla.gather(x, torch.arange(32, dtype=torch.int32, device="cuda"))
