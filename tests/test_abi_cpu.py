"""The C-ABI library loads, exports every entry point include/hla.h declares, and
rejects invalid arguments on the host before any HIP call (no GPU needed: every
call here fails validation, so nothing is launched)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2511_05832_amd as hla

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hla.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:hla_status|const char \*)\s*(hla_\w+)\s*\(", text, re.M)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(hla.LIB_PATH):
        pytest.fail("libhla.so is not built (run python -m paper_2511_05832_amd.build)")
    return hla.lib()


def test_header_declares_the_binding_names():
    assert declared_functions() == sorted(hla.EXPORTED)


def test_library_exports_every_declared_symbol(L):
    out = subprocess.run(["nm", "-D", "--defined-only", hla.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\s[TW]\s(hla_\w+)$", out, re.M))
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(L, name)


def test_version_and_empty_error(L):
    assert b"gfx950" in L.hla_version()


def status_and_msg(L, st):
    return st, L.hla_last_error().decode()


def test_hilbert_validation(L):
    """Any H x W grid up to 32768 per side; nothing to write is a no-op."""
    assert L.hla_hilbert_perm(96, 96, None, None, None) == hla.HLA_OK
    assert L.hla_hilbert_perm(56, 128, None, None, None) == hla.HLA_OK
    st, msg = status_and_msg(L, L.hla_hilbert_perm(0, 64, None, None, None))
    assert st == hla.HLA_ERR_INVALID_ARG and "positive" in msg
    st, _ = status_and_msg(L, L.hla_hilbert_perm(64, 40000, None, None, None))
    assert st == hla.HLA_ERR_UNSUPPORTED
    st, _ = status_and_msg(L, L.hla_hilbert_perm(64, 64, ctypes.c_void_p(2), None, None))
    assert st == hla.HLA_ERR_INVALID_ARG
    st, msg = status_and_msg(L, L.hla_hilbert_perm(8, 8, ctypes.c_void_p(0x1000),
                                                   ctypes.c_void_p(0x1000 + 64), None))
    assert st == hla.HLA_ERR_INVALID_ARG and "overlap" in msg


def test_permute_validation(L):
    vp = ctypes.c_void_p
    a, b, o = vp(0x10000), vp(0x20000), vp(0x30000)
    cases = [
        ((None, b, o, 1, 1, 64, 64, hla.HLA_BF16, None), hla.HLA_ERR_INVALID_ARG, "src"),
        ((a, vp(0x20008), o, 1, 1, 64, 64, hla.HLA_BF16, None), hla.HLA_ERR_INVALID_ARG, "aligned"),
        ((a, b, None, 1, 1, 64, 64, hla.HLA_BF16, None), hla.HLA_ERR_INVALID_ARG, "order"),
        ((a, b, o, 0, 1, 64, 64, hla.HLA_BF16, None), hla.HLA_ERR_INVALID_ARG, "positive"),
        ((a, b, o, 1, 1, 64, 3, hla.HLA_BF16, None), hla.HLA_ERR_UNSUPPORTED, "multiple of 4"),
        ((a, b, o, 1, 1, 64, 64, 7, None), hla.HLA_ERR_INVALID_ARG, "dtype"),
        ((a, vp(0x10000 + 4096), o, 1, 1, 64, 64, hla.HLA_BF16, None), hla.HLA_ERR_INVALID_ARG, "overlap"),
    ]
    for fn in (L.hla_gather, L.hla_scatter):
        for args, want, text in cases:
            st, msg = status_and_msg(L, fn(*args))
            assert st == want and text in msg, (args, st, msg)


def desc(kind, H, W, p0, p1=0):
    return hla.PatternDesc(hla.PATTERN_IDS[kind], H, W, p0, p1)


def test_block_mask_dims(L):
    nq, nk = ctypes.c_int32(), ctypes.c_int32()
    d = desc("hilbert_slide", 256, 256, 512)
    assert L.hla_block_mask_dims(ctypes.byref(d), 128, 64, ctypes.byref(nq), ctypes.byref(nk)) == 0
    assert (nq.value, nk.value) == (512, 1024)
    # ragged tilings: ceil(N / tile) per axis (3136 = 24.5 * 128 = 49 * 64; 63 < 64)
    for dd, tm, tn, want in [(desc("hilbert_slide", 56, 56, 24), 128, 64, (25, 49)),
                             (desc("rowmajor_slide", 7, 9, 1, 1), 64, 16, (1, 4))]:
        assert L.hla_block_mask_dims(ctypes.byref(dd), tm, tn, ctypes.byref(nq), ctypes.byref(nk)) == 0
        assert (nq.value, nk.value) == want
    bad = [
        (desc("hilbert_slide", 64, 64, 128), 96, 64, hla.HLA_ERR_UNSUPPORTED),     # not pow2
        (desc("hilbert_slide", 64, 64, -1), 128, 64, hla.HLA_ERR_INVALID_ARG),
        (desc("hilbert_window", 64, 64, 0), 128, 64, hla.HLA_ERR_INVALID_ARG),
        (desc("hilbert_shifted_window", 64, 64, 16, 16), 128, 64, hla.HLA_ERR_INVALID_ARG),
        (desc("rowmajor_neighborhood", 64, 64, 65, 3), 128, 64, hla.HLA_ERR_INVALID_ARG),
        (desc("hilbert_neighborhood", 8, 8, 65), 16, 16, hla.HLA_ERR_INVALID_ARG),
        (hla.PatternDesc(42, 64, 64, 1, 1), 128, 64, hla.HLA_ERR_INVALID_ARG),
        (desc("hilbert_window", 0, 64, 4), 128, 64, hla.HLA_ERR_INVALID_ARG),
        (desc("hilbert_slide", 64, 64, 128), 2048, 64, hla.HLA_ERR_UNSUPPORTED),
    ]
    for d, tm, tn, want in bad:
        st = L.hla_block_mask_dims(ctypes.byref(d), tm, tn, ctypes.byref(nq), ctypes.byref(nk))
        assert st == want, (d.pattern, tm, tn, st, L.hla_last_error())


def test_build_block_mask_rejects_null_arrays(L):
    m = hla.BlockMaskStruct()
    m.pat = desc("hilbert_slide", 64, 64, 128)
    m.tile_m, m.tile_n = 128, 64
    assert L.hla_build_block_mask(ctypes.byref(m), None) == hla.HLA_ERR_INVALID_ARG
    assert "n_full" in L.hla_last_error().decode()
    assert L.hla_build_block_mask(None, None) == hla.HLA_ERR_INVALID_ARG


def fake_mask(kind="hilbert_slide", H=64, W=64, p0=128, tm=128, tn=64):
    m = hla.BlockMaskStruct()
    m.pat = desc(kind, H, W, p0)
    m.tile_m, m.tile_n = tm, tn
    m.N = H * W
    m.n_qtiles, m.n_ktiles = H * W // tm, H * W // tn
    m.n_full = m.full_idx = m.n_part = m.part_idx = 0x40000
    return m


def test_attn_validation(L):
    vp = ctypes.c_void_p
    q, k, v, o = vp(0x100000), vp(0x200000), vp(0x300000), vp(0x400000)
    N = 4096

    def call(m, d=64, dt=hla.HLA_BF16, scale=0.125, N_=N, out=o, B=2, heads=4):
        return L.hla_attn_fwd(q, k, v, ctypes.byref(m), out, None, B, heads, N_, d, dt, scale, None)

    m = fake_mask()
    assert call(m, d=48) == hla.HLA_ERR_UNSUPPORTED
    assert call(m, d=128) == hla.HLA_ERR_UNSUPPORTED
    assert call(m, N_=2048) == hla.HLA_ERR_INVALID_ARG and "built for" in L.hla_last_error().decode()
    assert call(m, scale=0.0) == hla.HLA_ERR_INVALID_ARG
    assert call(m, scale=float("nan")) == hla.HLA_ERR_INVALID_ARG
    assert call(m, dt=5) == hla.HLA_ERR_INVALID_ARG
    assert call(m, out=vp(0x100000 + 4096)) == hla.HLA_ERR_INVALID_ARG
    assert call(m, out=vp(0x400004)) == hla.HLA_ERR_INVALID_ARG
    assert call(fake_mask(tm=64, tn=128)) == hla.HLA_ERR_UNSUPPORTED
    assert call(fake_mask(tm=256, tn=64)) == hla.HLA_ERR_UNSUPPORTED
    m0 = fake_mask()
    m0.n_part = 0
    assert call(m0) == hla.HLA_ERR_INVALID_ARG
    assert L.hla_attn_fwd(q, k, v, None, o, None, 2, 4, N, 64, hla.HLA_BF16, 0.1, None) == hla.HLA_ERR_INVALID_ARG


def test_attn_fwd_perm_validation(L):
    """The fused-reordering forward checks its order array first, then everything
    hla_attn_fwd checks; every call here is invalid, so nothing is launched."""
    vp = ctypes.c_void_p
    q, k, v, o = vp(0x100000), vp(0x200000), vp(0x300000), vp(0x400000)
    N = 4096

    def call(order, m=None, d=64, scale=0.125):
        m = m or fake_mask()
        return L.hla_attn_fwd_perm(q, k, v, order, ctypes.byref(m), o, None, 2, 4, N, d,
                                   hla.HLA_BF16, scale, None)

    assert call(None) == hla.HLA_ERR_INVALID_ARG and "order" in L.hla_last_error().decode()
    assert call(vp(0x800004)) == hla.HLA_ERR_INVALID_ARG and "16-byte" in L.hla_last_error().decode()
    assert call(vp(0x100000 + 1024)) == hla.HLA_ERR_INVALID_ARG and "overlap" in L.hla_last_error().decode()
    assert call(vp(0x800000), d=48) == hla.HLA_ERR_UNSUPPORTED
    assert call(vp(0x800000), scale=0.0) == hla.HLA_ERR_INVALID_ARG
    assert call(vp(0x800000), m=fake_mask(tm=256, tn=64)) == hla.HLA_ERR_UNSUPPORTED


def test_attn_fwd_hilbert_validation(L):
    """The forward that computes its own Hilbert rows and tile lists takes only the
    Hilbert patterns on 2^k x 2^k grids, in bf16; every call here is invalid or
    unsupported, so nothing is launched."""
    vp = ctypes.c_void_p
    q, k, v, o = vp(0x100000), vp(0x200000), vp(0x300000), vp(0x400000)

    def call(kind="hilbert_slide", H=64, W=64, p0=128, p1=0, tm=128, tn=64, N=None, d=64,
             dt=hla.HLA_BF16, out=o):
        pat = hla.PatternDesc(hla.PATTERN_IDS[kind], H, W, p0, p1)
        n = H * W if N is None else N
        return L.hla_attn_fwd_hilbert(q, k, v, ctypes.byref(pat), tm, tn, out, None, 2, 4, n, d,
                                      dt, 0.125, None)

    def err():
        return L.hla_last_error().decode()

    assert L.hla_attn_fwd_hilbert(q, k, v, None, 128, 64, o, None, 2, 4, 4096, 64, hla.HLA_BF16,
                                  0.125, None) == hla.HLA_ERR_INVALID_ARG
    assert call(kind="rowmajor_window", p0=16, p1=16) == hla.HLA_ERR_UNSUPPORTED and "Hilbert patterns" in err()
    assert call(kind="rowmajor_slide", p0=4, p1=4) == hla.HLA_ERR_UNSUPPORTED
    assert call(H=64, W=32) == hla.HLA_ERR_UNSUPPORTED and "2^k" in err()
    assert call(H=96, W=96) == hla.HLA_ERR_UNSUPPORTED
    assert call(H=2, W=2, p0=1) == hla.HLA_ERR_UNSUPPORTED
    assert call(H=4, W=4, p0=4) == hla.HLA_ERR_UNSUPPORTED and ">= 8" in err()
    assert call(dt=hla.HLA_F32) == hla.HLA_ERR_UNSUPPORTED and "bf16" in err()
    assert call(N=2048) == hla.HLA_ERR_INVALID_ARG and "built for" in err()
    assert call(d=48) == hla.HLA_ERR_UNSUPPORTED
    assert call(tm=64, tn=128) == hla.HLA_ERR_UNSUPPORTED
    assert call(tm=100) == hla.HLA_ERR_UNSUPPORTED
    assert call(out=vp(0x100000 + 4096)) == hla.HLA_ERR_INVALID_ARG
    assert call(kind="hilbert_window", p0=0) == hla.HLA_ERR_INVALID_ARG


def test_attn_fwd_rpb_validation(L):
    """Every call here is invalid, so nothing is launched."""
    vp = ctypes.c_void_p
    q, k, v, o = vp(0x100000), vp(0x200000), vp(0x300000), vp(0x400000)
    N = 4096

    def call(order, rpb, m=None, d=64):
        m = m or fake_mask()
        return L.hla_attn_fwd_rpb(q, k, v, order, rpb, ctypes.byref(m), o, None, 2, 4, N, d,
                                  hla.HLA_BF16, 0.125, None)

    good_o, good_t = vp(0x800000), vp(0x900000)
    assert call(None, good_t) == hla.HLA_ERR_INVALID_ARG and "order" in L.hla_last_error().decode()
    assert call(vp(0x800004), good_t) == hla.HLA_ERR_INVALID_ARG
    assert call(good_o, None) == hla.HLA_ERR_INVALID_ARG and "rpb" in L.hla_last_error().decode()
    assert call(good_o, vp(0x900002)) == hla.HLA_ERR_INVALID_ARG
    assert call(good_o, vp(0x100000 + 64)) == hla.HLA_ERR_INVALID_ARG and "overlap" in L.hla_last_error().decode()
    assert call(good_o, good_t, d=48) == hla.HLA_ERR_UNSUPPORTED


def test_build_path_and_mask_validation(L):
    """Both halves are validated before anything is enqueued; the mask must be on
    the path's grid and the outputs may not overlap its arrays."""
    vp = ctypes.c_void_p
    m = fake_mask(H=64, W=64)
    order, rank = vp(0x1000000), vp(0x2000000)
    assert L.hla_build_path_and_mask(64, 32, order, rank, ctypes.byref(m), None) == hla.HLA_ERR_INVALID_ARG
    assert "grid" in L.hla_last_error().decode()
    assert L.hla_build_path_and_mask(0, 64, order, rank, ctypes.byref(m), None) == hla.HLA_ERR_INVALID_ARG
    assert L.hla_build_path_and_mask(64, 64, vp(0x1000002), rank, ctypes.byref(m), None) == hla.HLA_ERR_INVALID_ARG
    assert L.hla_build_path_and_mask(64, 64, order, vp(0x1000000 + 64), ctypes.byref(m), None) == hla.HLA_ERR_INVALID_ARG
    assert L.hla_build_path_and_mask(64, 64, order, rank, None, None) == hla.HLA_ERR_INVALID_ARG
    assert L.hla_build_path_and_mask(64, 64, vp(m.full_idx + 8), rank, ctypes.byref(m), None) == hla.HLA_ERR_INVALID_ARG
    assert "overlaps" in L.hla_last_error().decode()
    m.n_full_t = 0x60000      # one of four transposed-list pointers
    assert L.hla_build_path_and_mask(64, 64, order, rank, ctypes.byref(m), None) == hla.HLA_ERR_INVALID_ARG
    bad = fake_mask(H=64, W=64, tm=2048)
    assert L.hla_build_path_and_mask(64, 64, order, rank, ctypes.byref(bad), None) == hla.HLA_ERR_UNSUPPORTED


def test_build_block_mask_rejects_partial_column_lists(L):
    m = hla.BlockMaskStruct()
    m.pat = desc("hilbert_slide", 64, 64, 128)
    m.tile_m, m.tile_n = 128, 64
    m.n_full = m.full_idx = m.n_part = m.part_idx = 0x40000
    m.n_full_t = m.full_idx_t = 0x50000
    assert L.hla_build_block_mask(ctypes.byref(m), None) == hla.HLA_ERR_INVALID_ARG
    assert "transposed" in L.hla_last_error().decode()
    m.n_part_t, m.part_idx_t = 0x50000, 0x50002
    assert L.hla_build_block_mask(ctypes.byref(m), None) == hla.HLA_ERR_INVALID_ARG
    assert "part_idx_t" in L.hla_last_error().decode()


def test_attn_bwd_validation(L):
    """Every call here is invalid, so nothing is launched."""
    vp = ctypes.c_void_p
    N, B, heads, d = 4096, 2, 4, 64
    tensor = B * heads * N * d * 2
    base = [vp(0x10000000 + i * 0x1000000) for i in range(10)]   # 16 MiB apart > tensor
    assert tensor <= 0x1000000
    q, k, v, o, g, lse, dq, dk, dv, st = base

    def call(m, **kw):
        a = dict(q=q, k=k, v=v, out=o, dout=g, lse=lse, dq=dq, dk=dk, dv=dv, stats=st,
                 d=d, dt=hla.HLA_BF16, scale=0.125, N=N)
        a.update(kw)
        return L.hla_attn_bwd(a["q"], a["k"], a["v"], a["out"], a["dout"], a["lse"],
                              ctypes.byref(m) if m is not None else None, a["dq"], a["dk"],
                              a["dv"], a["stats"], B, heads, a["N"], a["d"], a["dt"],
                              a["scale"], None)

    m = fake_mask()
    assert call(m) == hla.HLA_ERR_INVALID_ARG          # no transposed lists
    assert "transposed" in L.hla_last_error().decode()
    m.n_full_t = m.full_idx_t = m.n_part_t = m.part_idx_t = 0x60000
    assert call(None) == hla.HLA_ERR_INVALID_ARG
    assert call(m, d=48) == hla.HLA_ERR_UNSUPPORTED
    assert call(m, N=2048) == hla.HLA_ERR_INVALID_ARG
    assert call(m, scale=-1.0) == hla.HLA_ERR_INVALID_ARG
    assert call(m, lse=None) == hla.HLA_ERR_INVALID_ARG
    assert call(m, stats=None) == hla.HLA_ERR_INVALID_ARG
    assert call(m, dout=vp(0x10000008)) == hla.HLA_ERR_INVALID_ARG      # misaligned
    assert call(m, dk=vp(q.value + 4096)) == hla.HLA_ERR_INVALID_ARG     # dk overlaps q
    assert "overlaps" in L.hla_last_error().decode()
    assert call(m, dv=vp(dq.value + 64)) == hla.HLA_ERR_INVALID_ARG      # dv overlaps dq
    assert call(m, stats=vp(dv.value + 256)) == hla.HLA_ERR_INVALID_ARG  # stats overlaps dv
    assert call(m, stats=vp(lse.value)) == hla.HLA_ERR_INVALID_ARG       # stats overlaps lse
    assert call(fake_mask(tm=256, tn=64)) == hla.HLA_ERR_UNSUPPORTED


def test_attn_bwd_perm_validation(L):
    """The fused-reordering backward checks its order array, then everything
    hla_attn_bwd checks; every call here is invalid, so nothing is launched."""
    vp = ctypes.c_void_p
    N, B, heads, d = 4096, 2, 4, 64
    base = [vp(0x10000000 + i * 0x1000000) for i in range(11)]
    q, k, v, o, g, lse, dq, dk, dv, st, order = base
    m = fake_mask()
    m.n_full_t = m.full_idx_t = m.n_part_t = m.part_idx_t = 0x60000

    def call(**kw):
        a = dict(order=order, dq=dq, d=d)
        a.update(kw)
        return L.hla_attn_bwd_perm(q, k, v, o, g, lse, a["order"], ctypes.byref(m), a["dq"], dk, dv,
                                   st, B, heads, N, a["d"], hla.HLA_BF16, 0.125, None)

    assert call(order=None) == hla.HLA_ERR_INVALID_ARG and "order" in L.hla_last_error().decode()
    assert call(order=vp(order.value + 4)) == hla.HLA_ERR_INVALID_ARG and "16-byte" in L.hla_last_error().decode()
    assert call(order=vp(dq.value + 4096)) == hla.HLA_ERR_INVALID_ARG and "overlap" in L.hla_last_error().decode()
    assert call(d=48) == hla.HLA_ERR_UNSUPPORTED


def test_attn_bwd_noalloc_validation(L):
    """The allocation-free backward checks what hla_attn_bwd checks (less the stats
    workspace it does not take), and rejects more than 2^20 (b, h, row) rows, the
    capacity of its own array; every call here is invalid, so nothing is launched
    and no HIP call is made."""
    vp = ctypes.c_void_p
    N, d = 4096, 64
    base = [vp(0x100000000 + i * 0x10000000) for i in range(9)]   # 256 MiB apart
    q, k, v, o, g, lse, dq, dk, dv = base
    m = fake_mask()

    def call(mask, B=2, heads=4, **kw):
        a = dict(q=q, dq=dq, dk=dk, d=d, scale=0.125)
        a.update(kw)
        return L.hla_attn_bwd_noalloc(a["q"], k, v, o, g, lse, ctypes.byref(mask), a["dq"], a["dk"],
                                      dv, B, heads, N, a["d"], hla.HLA_BF16, a["scale"], None)

    assert call(m) == hla.HLA_ERR_INVALID_ARG and "transposed" in L.hla_last_error().decode()
    m.n_full_t = m.full_idx_t = m.n_part_t = m.part_idx_t = 0x60000
    assert call(m, q=None) == hla.HLA_ERR_INVALID_ARG
    assert call(m, d=48) == hla.HLA_ERR_UNSUPPORTED
    assert call(m, scale=0.0) == hla.HLA_ERR_INVALID_ARG
    assert call(m, dk=vp(dq.value + 64)) == hla.HLA_ERR_INVALID_ARG and "overlaps" in L.hla_last_error().decode()
    # 2 x 129 x 4096 = 1056768 rows > 2^20 (each tensor 129 MiB, inside the spacing)
    assert call(m, B=2, heads=129) == hla.HLA_ERR_UNSUPPORTED
    assert "exceeds" in L.hla_last_error().decode()


def test_proj_validation(L):
    vp = ctypes.c_void_p
    x, w, q, k, v = (vp(0x100000 * i) for i in range(1, 6))
    assert L.hla_qkv_proj(x, w, q, k, v, 16, 4096, 6, 48, None) == hla.HLA_ERR_UNSUPPORTED
    assert L.hla_qkv_proj(x, w, q, k, v, 16, 4096, 3, 32, None) == hla.HLA_ERR_UNSUPPORTED  # C = 96
    assert L.hla_qkv_proj(None, w, q, k, v, 16, 4096, 6, 32, None) == hla.HLA_ERR_INVALID_ARG
    assert L.hla_qkv_proj(x, w, q, k, v, 0, 4096, 6, 32, None) == hla.HLA_ERR_INVALID_ARG
    assert L.hla_out_proj(x, w, q, 16, 4096, 6, 32, 100, None) == hla.HLA_ERR_UNSUPPORTED
    assert L.hla_out_proj(x, w, vp(0x300008), 16, 4096, 6, 32, 192, None) == hla.HLA_ERR_INVALID_ARG


def test_proj_perm_validation(L):
    """The reordering variants: the plain projections' checks plus a null or
    misaligned order, all rejected on the host before any GPU call."""
    vp = ctypes.c_void_p
    x, w, q, k, v = (vp(0x100000 * i) for i in range(1, 6))
    order = vp(0x700000)
    assert L.hla_qkv_proj_perm(x, w, order, q, k, v, 16, 4096, 6, 48, None) == hla.HLA_ERR_UNSUPPORTED
    assert L.hla_qkv_proj_perm(x, w, None, q, k, v, 16, 4096, 6, 32, None) == hla.HLA_ERR_INVALID_ARG
    assert L.hla_qkv_proj_perm(x, w, vp(0x700004), q, k, v, 16, 4096, 6, 32, None) == hla.HLA_ERR_INVALID_ARG
    assert L.hla_qkv_proj_perm(None, w, order, q, k, v, 16, 4096, 6, 32, None) == hla.HLA_ERR_INVALID_ARG
    assert L.hla_out_proj_perm(x, w, order, q, 16, 4096, 6, 32, 100, None) == hla.HLA_ERR_UNSUPPORTED
    assert L.hla_out_proj_perm(x, w, None, q, 16, 4096, 6, 32, 192, None) == hla.HLA_ERR_INVALID_ARG
    assert L.hla_out_proj_perm(x, w, vp(0x700008), q, 16, 4096, 6, 32, 192, None) == hla.HLA_ERR_INVALID_ARG
    assert L.hla_out_proj_perm(x, w, order, q, 0, 4096, 6, 32, 192, None) == hla.HLA_ERR_INVALID_ARG


def test_binding_fails_loudly_without_gpu_tensors():
    import torch
    x = torch.zeros(2, 4, 64, 64, dtype=torch.bfloat16)
    order = torch.arange(64, dtype=torch.int32)
    with pytest.raises(hla.HLAError):
        hla.gather(x, order)
