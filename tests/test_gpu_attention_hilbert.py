"""GPU parity of the forward that computes its own Hilbert rows and tile lists
(hla_attn_fwd_hilbert).

It runs the fused-reordering forward's arithmetic on the same rows and tiles in
the same order, so it must equal hla_hilbert_perm -> hla_build_block_mask ->
hla_attn_fwd_perm bit for bit (that path is itself checked against the oracle,
tests/test_gpu_attention_perm.py). One small case per pattern kind is also checked
against the oracle directly, at the plain forward's bars.
"""
import zlib

import numpy as np
import pytest
import torch

import paper_2511_05832_amd as hla
import workloads as W
from conftest import Pat
from helpers import DEV, TOL_LSE, TOL_OUT, max_abs, np64
from oracle import attention as o_attn
from oracle import hilbert as o_hil
from oracle import permute as o_perm

pytestmark = pytest.mark.gpu


def both(pattern, tile_m, B, heads, d, seed, scale=None):
    q, k, v = (t.to(DEV) for t in W.attn_inputs(B, heads, pattern.N, d, "bf16", seed))
    scale = scale if scale is not None else 1.0 / d ** 0.5
    out_h, lse_h = hla.attn_fwd_hilbert(q, k, v, pattern, tile_m, 64, scale)
    order, _ = hla.hilbert_perm(pattern.H, pattern.W)
    mask = hla.build_block_mask(pattern, tile_m, 64)
    out_p, lse_p = hla.attn_fwd_perm(q, k, v, order, mask, scale)
    torch.cuda.synchronize()
    assert torch.equal(out_h, out_p), f"{pattern} tile {tile_m}: out differs from the precomputed path"
    assert torch.equal(lse_h, lse_p), f"{pattern} tile {tile_m}: lse differs from the precomputed path"
    return q, k, v, out_h, lse_h, scale


# every Hilbert pattern kind, parameters that put tile edges inside and across
# windows and bands, both tile heights, both head dims; grids 8x8 .. 64x64 (8x8
# is smaller than a 128-row tile: one ragged query-tile row)
CASES = [
    (Pat("hilbert_window", 32, 32, 64), 128, 64),
    (Pat("hilbert_window", 32, 32, 64), 64, 32),
    (Pat("hilbert_window", 64, 64, 256), 128, 64),
    (Pat("hilbert_window", 32, 32, 48), 128, 64),
    (Pat("hilbert_window", 16, 16, 16), 64, 64),
    (Pat("hilbert_window", 32, 32, 1024), 128, 32),
    (Pat("hilbert_slide", 32, 32, 64), 128, 64),
    (Pat("hilbert_slide", 64, 64, 128), 128, 64),
    (Pat("hilbert_slide", 64, 64, 64), 64, 32),
    (Pat("hilbert_slide", 32, 32, 5), 128, 64),
    (Pat("hilbert_slide", 32, 32, 2000), 64, 64),
    (Pat("hilbert_neighborhood", 32, 32, 81), 128, 64),
    (Pat("hilbert_neighborhood", 32, 32, 289), 64, 32),
    (Pat("hilbert_neighborhood", 16, 16, 256), 128, 64),
    (Pat("hilbert_shifted_window", 32, 32, 64, 32), 128, 64),
    (Pat("hilbert_shifted_window", 32, 32, 64, 5), 64, 64),
    (Pat("hilbert_shifted_window", 32, 32, 256, 200), 128, 32),
    (Pat("hilbert_shifted_window", 16, 16, 16, 4), 64, 64),
    (Pat("hilbert_slide", 8, 8, 9), 128, 64),
    (Pat("hilbert_neighborhood", 8, 8, 25), 64, 64),
]


@pytest.mark.parametrize("pat,tile_m,d", CASES, ids=lambda x: str(x) if isinstance(x, Pat) else None)
def test_equals_precomputed_index_and_lists(pat, tile_m, d):
    both(pat, tile_m, 2, 3, d, seed=zlib.crc32(repr(pat).encode()) % 1000 + tile_m + d)


@pytest.mark.parametrize("kind,p0,p1", [("hilbert_window", 64, 0), ("hilbert_slide", 40, 0),
                                        ("hilbert_neighborhood", 49, 0),
                                        ("hilbert_shifted_window", 64, 16)])
def test_against_the_oracle(kind, p0, p1):
    pat = Pat(kind, 16, 16, p0, p1)
    q, k, v, out, lse, scale = both(pat, 128, 1, 2, 64, seed=7)
    order = o_hil.hilbert_order(pat.H, pat.W)
    qn, kn, vn = (o_perm.gather(np64(t), order) for t in (q, k, v))
    ref_out, ref_lse = o_attn.attention(qn, kn, vn, pat, scale)
    got_out = o_perm.gather(np64(out), order)
    got_lse = np64(lse)[:, :, order]
    assert max_abs(got_out, ref_out) <= TOL_OUT["bf16"]
    assert max_abs(got_lse, ref_lse) <= TOL_LSE


@pytest.mark.parametrize("name", ["hsa_bf16_64x64_h128", "hwa_bf16_128x128_w256", "hsa_bf16_256x256_h512"])
def test_full_size_workloads(name):
    w = W.WORKLOADS[name]
    both(w.pattern, w.tile_m, w.B, w.heads, w.d, seed=w.seed, scale=w.scale)


# several heads per workgroup (the launcher picks more than one only for large
# grids; the override forces it): head counts that do and do not divide B*heads,
# rows with one key tile (window = tile) and with many
@pytest.mark.parametrize("hpw", [1, 2, 3, 4, 7])
@pytest.mark.parametrize("pat,tile_m,d", [
    (Pat("hilbert_window", 32, 32, 64), 64, 64),
    (Pat("hilbert_window", 16, 16, 16), 64, 32),
    (Pat("hilbert_slide", 32, 32, 64), 128, 64),
    (Pat("hilbert_shifted_window", 32, 32, 256, 200), 128, 32),
    (Pat("hilbert_neighborhood", 8, 8, 25), 128, 64),
], ids=lambda x: str(x) if isinstance(x, Pat) else None)
def test_heads_per_workgroup(monkeypatch, hpw, pat, tile_m, d):
    monkeypatch.setenv("HLA_ATTN_HEADS_PER_WORKGROUP", str(hpw))
    both(pat, tile_m, 2, 3, d, seed=hpw * 31 + tile_m + d)


@pytest.mark.parametrize("value", ["0", "65", "abc", ""])
def test_heads_per_workgroup_override_out_of_range_is_ignored(monkeypatch, value):
    pat = Pat("hilbert_window", 32, 32, 64)
    q, k, v = (t.to(DEV) for t in W.attn_inputs(2, 3, pat.N, 64, "bf16", 9))
    monkeypatch.delenv("HLA_ATTN_HEADS_PER_WORKGROUP", raising=False)
    out_a, lse_a = hla.attn_fwd_hilbert(q, k, v, pat, 128, 64, 0.125)
    monkeypatch.setenv("HLA_ATTN_HEADS_PER_WORKGROUP", value)
    out_b, lse_b = hla.attn_fwd_hilbert(q, k, v, pat, 128, 64, 0.125)
    torch.cuda.synchronize()
    assert torch.equal(out_a, out_b) and torch.equal(lse_a, lse_b)


def test_heads_per_workgroup_without_lse(monkeypatch):
    monkeypatch.setenv("HLA_ATTN_HEADS_PER_WORKGROUP", "4")
    pat = Pat("hilbert_slide", 32, 32, 64)
    q, k, v = (t.to(DEV) for t in W.attn_inputs(2, 3, pat.N, 64, "bf16", 5))
    out_a, _ = hla.attn_fwd_hilbert(q, k, v, pat, 128, 64, 0.125)
    out_b, lse_b = hla.attn_fwd_hilbert(q, k, v, pat, 128, 64, 0.125, with_lse=False)
    torch.cuda.synchronize()
    assert lse_b is None and torch.equal(out_a, out_b)


# rows listing more key tiles than the kernel's block table holds (256): the
# entries past it walk the curve per tile
@pytest.mark.parametrize("pat,tile_m,d", [(Pat("hilbert_slide", 256, 256, 20000), 128, 32),
                                          (Pat("hilbert_window", 256, 256, 32768), 64, 32),
                                          (Pat("hilbert_neighborhood", 256, 256, 40000), 128, 64),
                                          (Pat("hilbert_shifted_window", 256, 256, 24576, 5000), 128, 32),
                                          (Pat("hilbert_slide", 512, 512, 9000), 128, 32)],
                         ids=lambda x: str(x) if isinstance(x, Pat) else None)
def test_rows_longer_than_the_block_table(pat, tile_m, d):
    both(pat, tile_m, 1, 1, d, seed=zlib.crc32(repr(pat).encode()) % 1000)


def test_layer_attention_shape():
    """The layer's attention: 64x64 grid, band +-64, B=16, 6 heads of 32, 64x64 tiles."""
    both(Pat("hilbert_slide", 64, 64, 64), 64, 16, 6, 32, seed=4, scale=32 ** -0.5)


def test_lse_may_be_omitted():
    pat = Pat("hilbert_slide", 32, 32, 64)
    q, k, v = (t.to(DEV) for t in W.attn_inputs(1, 2, pat.N, 64, "bf16", 3))
    out_a, _ = hla.attn_fwd_hilbert(q, k, v, pat, 128, 64, 0.125)
    out_b, lse_b = hla.attn_fwd_hilbert(q, k, v, pat, 128, 64, 0.125, with_lse=False)
    torch.cuda.synchronize()
    assert lse_b is None and torch.equal(out_a, out_b)
