"""GPU test of the allocation-free backward (hla_attn_bwd_noalloc), called through
the C ABI: its gradients equal hla_attn_bwd's (the same kernels, with the row
statistics in the library's own per-device array instead of a workspace) bit for
bit, on two calls in a row, the second with a smaller input, and on a call at the
array's largest size."""
import ctypes

import pytest
import torch

import paper_2511_05832_amd as hla
import workloads as W
from conftest import Pat

pytestmark = pytest.mark.gpu

MAX_ROWS = 1 << 20


def forward(pat, B, Hh, d, dtype, tm, seed):
    q, k, v = (t.cuda() for t in W.attn_inputs(B, Hh, pat.N, d, dtype, seed))
    g = torch.Generator().manual_seed(seed + 1)
    dout = torch.randn((B, Hh, pat.N, d), generator=g).to(q.dtype).cuda()
    mask = hla.BlockMask(pat, tm, 64, columns=True).build()
    out, lse = hla.attn_fwd(q, k, v, mask, 1.0 / d ** 0.5)
    return q, k, v, out, dout, lse, mask


def noalloc_through_the_abi(q, k, v, out, dout, lse, mask, scale):
    B, Hh, N, d = q.shape
    dq, dk, dv = (torch.full_like(q, float("nan")) for _ in range(3))
    st = hla.lib().hla_attn_bwd_noalloc(
        hla._ptr(q), hla._ptr(k), hla._ptr(v), hla._ptr(out), hla._ptr(dout), hla._ptr(lse),
        ctypes.byref(mask.struct), hla._ptr(dq), hla._ptr(dk), hla._ptr(dv), B, Hh, N, d,
        hla._dtype_code(q), scale, hla._stream(q))
    assert st == hla.HLA_OK, hla.lib().hla_last_error().decode()
    return dq, dk, dv


def check_case(pat, B, Hh, d, dtype, tm, seed):
    q, k, v, out, dout, lse, mask = forward(pat, B, Hh, d, dtype, tm, seed)
    scale = 1.0 / d ** 0.5
    got = noalloc_through_the_abi(q, k, v, out, dout, lse, mask, scale)
    want = hla.attn_bwd(q, k, v, out, dout, lse, mask, scale)
    torch.cuda.synchronize()
    print(f"{pat} B={B} heads={Hh} d={d} {dtype}: rows {B * Hh * pat.N}", flush=True)
    for g_, w_, name in zip(got, want, ("dq", "dk", "dv")):
        assert torch.equal(g_, w_), f"{name} differs from hla_attn_bwd"


def test_two_calls_in_a_row_second_smaller():
    # first: a 64 x 64 band, 2 x 4 slices (32768 rows); second: a 32 x 32 window,
    # 1 x 2 slices (2048 rows), another pattern, head_dim and dtype, so that any
    # statistics left from the first call would show
    check_case(Pat("hilbert_slide", 64, 64, 128), 2, 4, 64, "bf16", 128, 41)
    check_case(Pat("hilbert_window", 32, 32, 64), 1, 2, 32, "f32", 64, 42)


def test_largest_size_then_a_small_one():
    # B * heads * N = 2^20, the array's capacity, then a ragged small call
    check_case(Pat("hilbert_slide", 256, 256, 512), 2, 8, 64, "bf16", 128, 43)
    check_case(Pat("rowmajor_slide", 9, 21, 2, 3), 1, 3, 64, "bf16", 64, 44)


def test_rejects_more_rows_than_the_array_holds():
    pat = Pat("hilbert_window", 64, 64, 256)
    q, k, v, out, dout, lse, mask = forward(pat, 1, 1, 64, "bf16", 128, 45)
    B, Hh, N, d = 1, MAX_ROWS // pat.N + 1, pat.N, 64
    big = [torch.empty((B, Hh, N, d), dtype=torch.bfloat16, device="cuda") for _ in range(8)]
    lse_big = torch.empty((B, Hh, N), dtype=torch.float32, device="cuda")
    st = hla.lib().hla_attn_bwd_noalloc(
        *(hla._ptr(t) for t in big[:5]), hla._ptr(lse_big), ctypes.byref(mask.struct),
        *(hla._ptr(t) for t in big[5:]), B, Hh, N, d, hla.HLA_BF16, 0.125, hla._stream(q))
    assert st == hla.HLA_ERR_UNSUPPORTED
    assert "exceeds" in hla.lib().hla_last_error().decode()
    # the array is untouched by a rejected call: a valid call still matches
    check_case(pat, 1, 2, 64, "bf16", 128, 46)
