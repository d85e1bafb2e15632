"""Python binding of libhla: Hilbert-guided block-sparse local attention on MI355X.

Argument marshalling only. Every step runs in the HIP kernels of libhla.so
(see include/hla.h); torch supplies device buffers and the current stream. If
the library has not been built the first call raises ``HLAError`` - there is no
fallback path.

    order, rank = hilbert_perm(H, W)
    qh = gather(q, order)                       # into Hilbert order
    mask = build_block_mask(pattern, 128, 64)   # full / partial / empty tile lists
    out, lse = attn_fwd(qh, kh, vh, mask, scale)
    o = scatter(out, order)                     # back to row-major
    o, lse_rm = attn_fwd_perm(q, k, v, order, mask, scale)   # the same, reordering fused

    mask = build_block_mask(pattern, 128, 64, columns=True)   # + per-column lists
    dq, dk, dv = attn_bwd(qh, kh, vh, out, dout, lse, mask, scale)

Patterns are given as any object with attributes kind, H, W, p0, p1 (kind is one
of PATTERN_IDS), or as a tuple (kind, H, W, p0, p1).
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional, Tuple

import torch

__all__ = ["HLAError", "lib", "hilbert_perm", "gather", "scatter", "block_mask_dims",
           "build_block_mask", "BlockMask", "attn_fwd", "attn_fwd_perm", "attn_fwd_hilbert",
           "attn_fwd_rpb", "attn_bwd",
           "attn_bwd_perm",
           "qkv_proj", "out_proj",
           "PATTERN_IDS", "LIB_PATH", "EXPORTED"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhla.so")

PATTERN_IDS = {
    "hilbert_window": 0,
    "hilbert_slide": 1,
    "rowmajor_window": 2,
    "rowmajor_slide": 3,
    "hilbert_neighborhood": 4,
    "rowmajor_neighborhood": 5,
    "hilbert_shifted_window": 6,
}

HLA_OK, HLA_ERR_INVALID_ARG, HLA_ERR_UNSUPPORTED, HLA_ERR_HIP = 0, 1, 2, 3
HLA_F32, HLA_BF16 = 0, 1

EXPORTED = ("hla_hilbert_perm", "hla_gather", "hla_scatter", "hla_block_mask_dims",
            "hla_build_block_mask", "hla_build_path_and_mask", "hla_attn_fwd", "hla_attn_fwd_perm",
            "hla_attn_fwd_hilbert", "hla_attn_fwd_rpb",
            "hla_attn_bwd", "hla_attn_bwd_perm", "hla_attn_bwd_noalloc",
            "hla_qkv_proj", "hla_out_proj", "hla_qkv_proj_perm", "hla_out_proj_perm",
            "hla_last_error", "hla_version")


class HLAError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"[hla status {status}] {message}")
        self.status = status


class PatternDesc(ctypes.Structure):
    _fields_ = [("pattern", ctypes.c_int32), ("H", ctypes.c_int32), ("W", ctypes.c_int32),
                ("p0", ctypes.c_int32), ("p1", ctypes.c_int32)]


_i32p = ctypes.POINTER(ctypes.c_int32)


class BlockMaskStruct(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int32), ("tile_m", ctypes.c_int32), ("tile_n", ctypes.c_int32),
                ("n_qtiles", ctypes.c_int32), ("n_ktiles", ctypes.c_int32),
                ("pat", PatternDesc),
                ("n_full", ctypes.c_void_p), ("full_idx", ctypes.c_void_p),
                ("n_part", ctypes.c_void_p), ("part_idx", ctypes.c_void_p),
                ("totals", ctypes.c_void_p),
                ("n_full_t", ctypes.c_void_p), ("full_idx_t", ctypes.c_void_p),
                ("n_part_t", ctypes.c_void_p), ("part_idx_t", ctypes.c_void_p)]


_lib = None
_lib_lock = threading.Lock()


def lib() -> ctypes.CDLL:
    """Load libhla.so (once). Raises HLAError if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    with _lib_lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise HLAError(-1, f"{LIB_PATH} is not built; run `python -m paper_2511_05832_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
        sigs = {
            "hla_hilbert_perm": [i32, i32, vp, vp, vp],
            "hla_gather": [vp, vp, vp, i64, i64, i64, i64, ctypes.c_int, vp],
            "hla_scatter": [vp, vp, vp, i64, i64, i64, i64, ctypes.c_int, vp],
            "hla_block_mask_dims": [ctypes.POINTER(PatternDesc), i32, i32, _i32p, _i32p],
            "hla_build_block_mask": [ctypes.POINTER(BlockMaskStruct), vp],
            "hla_build_path_and_mask": [i32, i32, vp, vp, ctypes.POINTER(BlockMaskStruct), vp],
            "hla_attn_fwd": [vp, vp, vp, ctypes.POINTER(BlockMaskStruct), vp, vp,
                             i64, i64, i64, i64, ctypes.c_int, f32, vp],
            "hla_attn_fwd_perm": [vp, vp, vp, vp, ctypes.POINTER(BlockMaskStruct), vp, vp,
                                  i64, i64, i64, i64, ctypes.c_int, f32, vp],
            "hla_attn_fwd_hilbert": [vp, vp, vp, ctypes.POINTER(PatternDesc), i32, i32, vp, vp,
                                     i64, i64, i64, i64, ctypes.c_int, f32, vp],
            "hla_attn_fwd_rpb": [vp, vp, vp, vp, vp, ctypes.POINTER(BlockMaskStruct), vp, vp,
                                 i64, i64, i64, i64, ctypes.c_int, f32, vp],
            "hla_attn_bwd": [vp, vp, vp, vp, vp, vp, ctypes.POINTER(BlockMaskStruct), vp, vp, vp,
                             vp, i64, i64, i64, i64, ctypes.c_int, f32, vp],
            "hla_attn_bwd_perm": [vp, vp, vp, vp, vp, vp, vp, ctypes.POINTER(BlockMaskStruct), vp, vp,
                                  vp, vp, i64, i64, i64, i64, ctypes.c_int, f32, vp],
            "hla_attn_bwd_noalloc": [vp, vp, vp, vp, vp, vp, ctypes.POINTER(BlockMaskStruct), vp, vp,
                                     vp, i64, i64, i64, i64, ctypes.c_int, f32, vp],
            "hla_qkv_proj": [vp, vp, vp, vp, vp, i64, i64, i64, i64, vp],
            "hla_out_proj": [vp, vp, vp, i64, i64, i64, i64, i64, vp],
            "hla_qkv_proj_perm": [vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, vp],
            "hla_out_proj_perm": [vp, vp, vp, vp, i64, i64, i64, i64, i64, vp],
        }
        for name, args in sigs.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        L.hla_last_error.argtypes = []
        L.hla_last_error.restype = ctypes.c_char_p
        L.hla_version.argtypes = []
        L.hla_version.restype = ctypes.c_char_p
        _lib = L
        return _lib


def _check(status: int):
    if status != HLA_OK:
        raise HLAError(status, lib().hla_last_error().decode(errors="replace"))


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _ptr(t: Optional[torch.Tensor]):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return HLA_BF16
    if t.dtype == torch.float32:
        return HLA_F32
    raise HLAError(HLA_ERR_UNSUPPORTED, f"dtype {t.dtype} (supported: bfloat16, float32)")


def _require(t: torch.Tensor, name: str):
    if not isinstance(t, torch.Tensor):
        raise HLAError(HLA_ERR_INVALID_ARG, f"{name} must be a tensor")
    if t.device.type != "cuda":
        raise HLAError(HLA_ERR_INVALID_ARG, f"{name} must be on a GPU (got {t.device})")
    if not t.is_contiguous():
        raise HLAError(HLA_ERR_INVALID_ARG, f"{name} must be contiguous")


def _require_order(order: torch.Tensor, n: int):
    _require(order, "order")
    if order.dtype != torch.int32:
        raise HLAError(HLA_ERR_INVALID_ARG, "order must be int32")
    if order.numel() != n:
        raise HLAError(HLA_ERR_INVALID_ARG, f"order has {order.numel()} entries, expected {n}")


def _pattern_desc(pattern) -> PatternDesc:
    if isinstance(pattern, tuple):
        kind, H, W, p0, *rest = pattern
        p1 = rest[0] if rest else 0
    else:
        kind, H, W, p0, p1 = pattern.kind, pattern.H, pattern.W, pattern.p0, pattern.p1
    if kind not in PATTERN_IDS:
        raise HLAError(HLA_ERR_INVALID_ARG, f"unknown pattern kind {kind!r}")
    return PatternDesc(PATTERN_IDS[kind], int(H), int(W), int(p0), int(p1))


def hilbert_perm(H: int, W: int, device="cuda", out=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """(order, rank) int32 device tensors of length H*W (hla_hilbert_perm).
    ``out`` = (order, rank) preallocated tensors to write into."""
    if out is None:
        order = torch.empty(H * W, dtype=torch.int32, device=device)
        rank = torch.empty(H * W, dtype=torch.int32, device=device)
    else:
        order, rank = out
        for t, n in ((order, "order"), (rank, "rank")):
            _require(t, n)
            if t.dtype != torch.int32 or t.numel() != H * W:
                raise HLAError(HLA_ERR_INVALID_ARG, f"{n} must be int32 with H*W entries")
    _check(lib().hla_hilbert_perm(int(H), int(W), _ptr(order), _ptr(rank), _stream(order)))
    return order, rank


def _as4d(t: torch.Tensor):
    if t.dim() == 4:
        return t.shape
    if t.dim() == 3:      # [B, N, C] as heads = 1, d = C
        return (t.shape[0], 1, t.shape[1], t.shape[2])
    raise HLAError(HLA_ERR_INVALID_ARG, f"expected a [B, heads, N, d] or [B, N, C] tensor, got {tuple(t.shape)}")


def _permute(fn, src, order, out):
    _require(src, "src")
    _require(order, "order")
    if order.dtype != torch.int32:
        raise HLAError(HLA_ERR_INVALID_ARG, "order must be int32")
    B, Hh, N, d = _as4d(src)
    if order.numel() != N:
        raise HLAError(HLA_ERR_INVALID_ARG, f"order has {order.numel()} entries, tensor has N = {N}")
    if out is None:
        out = torch.empty_like(src)
    else:
        _require(out, "out")
        if out.shape != src.shape or out.dtype != src.dtype:
            raise HLAError(HLA_ERR_INVALID_ARG, "out must match src in shape and dtype")
    _check(fn(_ptr(src), _ptr(out), _ptr(order), B, Hh, N, d, _dtype_code(src), _stream(src)))
    return out


def gather(src: torch.Tensor, order: torch.Tensor, out: Optional[torch.Tensor] = None):
    """dst[..., i, :] = src[..., order[i], :] (hla_gather)."""
    return _permute(lib().hla_gather, src, order, out)


def scatter(src: torch.Tensor, order: torch.Tensor, out: Optional[torch.Tensor] = None):
    """dst[..., order[i], :] = src[..., i, :] (hla_scatter)."""
    return _permute(lib().hla_scatter, src, order, out)


def block_mask_dims(pattern, tile_m: int, tile_n: int) -> Tuple[int, int]:
    desc = _pattern_desc(pattern)
    nq, nk = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().hla_block_mask_dims(ctypes.byref(desc), int(tile_m), int(tile_n),
                                     ctypes.byref(nq), ctypes.byref(nk)))
    return nq.value, nk.value


class BlockMask:
    """Device tile lists of one (pattern, tile) pair; owns its buffers.

    ``columns=True`` also allocates and builds the per-key-tile-column lists
    that the backward pass walks."""

    def __init__(self, pattern, tile_m: int, tile_n: int, device="cuda", columns: bool = False,
                 totals: bool = True):
        nq, nk = block_mask_dims(pattern, tile_m, tile_n)
        self.pattern = pattern
        self.tile_m, self.tile_n, self.n_qtiles, self.n_ktiles = tile_m, tile_n, nq, nk
        self.n_full = torch.empty(nq, dtype=torch.int32, device=device)
        self.n_part = torch.empty(nq, dtype=torch.int32, device=device)
        self.full_idx = torch.empty((nq, nk), dtype=torch.int32, device=device)
        self.part_idx = torch.empty((nq, nk), dtype=torch.int32, device=device)
        self.totals = torch.empty(2, dtype=torch.int32, device=device)
        self.struct = BlockMaskStruct()
        self.struct.pat = _pattern_desc(pattern)
        self.struct.tile_m, self.struct.tile_n = int(tile_m), int(tile_n)
        self.struct.n_full = self.n_full.data_ptr()
        self.struct.full_idx = self.full_idx.data_ptr()
        self.struct.n_part = self.n_part.data_ptr()
        self.struct.part_idx = self.part_idx.data_ptr()
        # totals=False: the build writes only the lists (the attention reads nothing
        # else); host_totals() then sums the per-row counts itself
        self.with_totals = totals
        self.struct.totals = self.totals.data_ptr() if totals else 0
        self.columns = columns
        if columns:
            self.n_full_t = torch.empty(nk, dtype=torch.int32, device=device)
            self.n_part_t = torch.empty(nk, dtype=torch.int32, device=device)
            self.full_idx_t = torch.empty((nk, nq), dtype=torch.int32, device=device)
            self.part_idx_t = torch.empty((nk, nq), dtype=torch.int32, device=device)
            self.struct.n_full_t = self.n_full_t.data_ptr()
            self.struct.full_idx_t = self.full_idx_t.data_ptr()
            self.struct.n_part_t = self.n_part_t.data_ptr()
            self.struct.part_idx_t = self.part_idx_t.data_ptr()

    def build(self):
        _check(lib().hla_build_block_mask(ctypes.byref(self.struct), _stream(self.n_full)))
        return self

    def build_with_path(self, order: Optional[torch.Tensor] = None,
                        rank: Optional[torch.Tensor] = None):
        """Build the lists and the Hilbert index of the pattern's grid together
        (hla_build_path_and_mask: one launch on 2^k x 2^k grids). order, rank:
        int32 [H*W] outputs, either may be None."""
        n = self.struct.pat.H * self.struct.pat.W
        for t, name in ((order, "order"), (rank, "rank")):
            if t is not None:
                _require(t, name)
                if t.dtype != torch.int32 or t.numel() != n:
                    raise HLAError(HLA_ERR_INVALID_ARG, f"{name} must be int32 with H*W entries")
        _check(lib().hla_build_path_and_mask(int(self.struct.pat.H), int(self.struct.pat.W),
                                             _ptr(order), _ptr(rank), ctypes.byref(self.struct),
                                             _stream(self.n_full)))
        return self

    @property
    def N(self) -> int:
        return self.struct.N

    def host_totals(self) -> Tuple[int, int]:
        if not self.with_totals:
            return int(self.n_full.sum().item()), int(self.n_part.sum().item())
        t = self.totals.cpu()
        return int(t[0]), int(t[1])


def build_block_mask(pattern, tile_m: int, tile_n: int, device="cuda",
                     columns: bool = False) -> BlockMask:
    """Classify all tiles and build the per-row lists (hla_build_block_mask);
    ``columns=True`` adds the per-column lists for the backward pass."""
    return BlockMask(pattern, tile_m, tile_n, device, columns).build()


def _attn_fwd_args(q, k, v, scale, out, lse, with_lse):
    for t, n in ((q, "q"), (k, "k"), (v, "v")):
        _require(t, n)
    if q.dim() != 4 or k.shape != q.shape or v.shape != q.shape:
        raise HLAError(HLA_ERR_INVALID_ARG, "q, k, v must all be [B, heads, N, d] of one shape")
    if k.dtype != q.dtype or v.dtype != q.dtype:
        raise HLAError(HLA_ERR_INVALID_ARG, "q, k, v must share a dtype")
    B, Hh, N, d = q.shape
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    if out is None:
        out = torch.empty_like(q)
    else:
        _require(out, "out")
    if lse is None and with_lse:
        lse = torch.empty((B, Hh, N), dtype=torch.float32, device=q.device)
    elif lse is not None:
        _require(lse, "lse")
    return B, Hh, N, d, float(scale), out, lse


def attn_fwd(q, k, v, mask: BlockMask, scale: Optional[float] = None,
             out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
             with_lse: bool = True):
    """Block-sparse attention forward (hla_attn_fwd). Returns (out, lse or None)."""
    B, Hh, N, d, scale, out, lse = _attn_fwd_args(q, k, v, scale, out, lse, with_lse)
    _check(lib().hla_attn_fwd(_ptr(q), _ptr(k), _ptr(v), ctypes.byref(mask.struct), _ptr(out),
                              _ptr(lse), B, Hh, N, d, _dtype_code(q), scale, _stream(q)))
    return out, lse


def attn_fwd_perm(q, k, v, order, mask: BlockMask, scale: Optional[float] = None,
                  out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                  with_lse: bool = True):
    """Attention forward on grid-ordered q, k, v with the reordering fused in
    (hla_attn_fwd_perm): sequence position i is row order[i]; out and lse come
    back in grid order. Returns (out, lse or None)."""
    _require(order, "order")
    if order.dtype != torch.int32:
        raise HLAError(HLA_ERR_INVALID_ARG, "order must be int32")
    B, Hh, N, d, scale, out, lse = _attn_fwd_args(q, k, v, scale, out, lse, with_lse)
    if order.numel() != N:
        raise HLAError(HLA_ERR_INVALID_ARG, f"order has {order.numel()} entries, expected N = {N}")
    _check(lib().hla_attn_fwd_perm(_ptr(q), _ptr(k), _ptr(v), _ptr(order), ctypes.byref(mask.struct),
                                   _ptr(out), _ptr(lse), B, Hh, N, d, _dtype_code(q), scale,
                                   _stream(q)))
    return out, lse


def attn_fwd_hilbert(q, k, v, pattern, tile_m: int, tile_n: int, scale: Optional[float] = None,
                     out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                     with_lse: bool = True):
    """attn_fwd_perm with the Hilbert order and the tile lists computed inside the
    kernel (hla_attn_fwd_hilbert): q, k, v in grid order, a Hilbert pattern on a
    2^k x 2^k grid. Returns (out, lse or None), in grid order."""
    B, Hh, N, d, scale, out, lse = _attn_fwd_args(q, k, v, scale, out, lse, with_lse)
    desc = _pattern_desc(pattern)
    _check(lib().hla_attn_fwd_hilbert(_ptr(q), _ptr(k), _ptr(v), ctypes.byref(desc), int(tile_m),
                                      int(tile_n), _ptr(out), _ptr(lse), B, Hh, N, d, _dtype_code(q),
                                      scale, _stream(q)))
    return out, lse


def attn_fwd_rpb(q, k, v, order, rpb, mask: BlockMask, scale: Optional[float] = None,
                 out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                 with_lse: bool = True):
    """Attention forward with the global relative position bias (hla_attn_fwd_rpb):
    q, k, v in sequence order; order[i] = grid (row-major) id of sequence position i
    (None: the identity, for row-major patterns); rpb = float32 [heads, 2H-1, 2W-1].
    Returns (out, lse or None)."""
    B, Hh, N, d, scale, out, lse = _attn_fwd_args(q, k, v, scale, out, lse, with_lse)
    if order is None:
        order = torch.arange(N, dtype=torch.int32, device=q.device)
    _require(order, "order")
    _require(rpb, "rpb")
    if order.dtype != torch.int32 or order.numel() != N:
        raise HLAError(HLA_ERR_INVALID_ARG, f"order must be int32 with N = {N} entries")
    H, W = mask.struct.pat.H, mask.struct.pat.W
    if rpb.dtype != torch.float32 or tuple(rpb.shape) != (Hh, 2 * H - 1, 2 * W - 1):
        raise HLAError(HLA_ERR_INVALID_ARG, f"rpb must be float32 [{Hh}, {2 * H - 1}, {2 * W - 1}]")
    _check(lib().hla_attn_fwd_rpb(_ptr(q), _ptr(k), _ptr(v), _ptr(order), _ptr(rpb),
                                  ctypes.byref(mask.struct), _ptr(out), _ptr(lse), B, Hh, N, d,
                                  _dtype_code(q), scale, _stream(q)))
    return out, lse


def _attn_bwd_args(q, k, v, out, dout, lse, scale, dq, dk, dv, stats):
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (out, "out"), (dout, "dout"), (lse, "lse")):
        _require(t, n)
    if q.dim() != 4 or any(t.shape != q.shape for t in (k, v, out, dout)):
        raise HLAError(HLA_ERR_INVALID_ARG, "q, k, v, out, dout must all be [B, heads, N, d] of one shape")
    if any(t.dtype != q.dtype for t in (k, v, out, dout)):
        raise HLAError(HLA_ERR_INVALID_ARG, "q, k, v, out, dout must share a dtype")
    B, Hh, N, d = q.shape
    if lse.dtype != torch.float32 or tuple(lse.shape) != (B, Hh, N):
        raise HLAError(HLA_ERR_INVALID_ARG, "lse must be float32 [B, heads, N]")
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    if stats is None:
        stats = torch.empty((B, Hh, N, 2), dtype=torch.float32, device=q.device)
    for t, n in ((dq, "dq"), (dk, "dk"), (dv, "dv"), (stats, "stats")):
        _require(t, n)
    return B, Hh, N, d, float(scale), dq, dk, dv, stats


def attn_bwd(q, k, v, out, dout, lse, mask: BlockMask, scale: Optional[float] = None,
             dq: Optional[torch.Tensor] = None, dk: Optional[torch.Tensor] = None,
             dv: Optional[torch.Tensor] = None, stats: Optional[torch.Tensor] = None):
    """Block-sparse attention backward (hla_attn_bwd). ``out`` and ``lse`` are the
    forward's results for these q, k, v, mask and scale. Returns (dq, dk, dv).
    ``stats`` is the float32 [B, heads, N, 2] workspace (allocated if None)."""
    B, Hh, N, d, scale, dq, dk, dv, stats = _attn_bwd_args(q, k, v, out, dout, lse, scale,
                                                           dq, dk, dv, stats)
    _check(lib().hla_attn_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(lse),
                              ctypes.byref(mask.struct), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(stats),
                              B, Hh, N, d, _dtype_code(q), scale, _stream(q)))
    return dq, dk, dv


def attn_bwd_perm(q, k, v, out, dout, lse, order, mask: BlockMask, scale: Optional[float] = None,
                  dq: Optional[torch.Tensor] = None, dk: Optional[torch.Tensor] = None,
                  dv: Optional[torch.Tensor] = None, stats: Optional[torch.Tensor] = None):
    """Backward with the reordering fused in (hla_attn_bwd_perm): every tensor in grid
    order, sequence position i is row order[i]; ``out`` and ``lse`` are attn_fwd_perm's
    results. Returns (dq, dk, dv) in grid order."""
    B, Hh, N, d, scale, dq, dk, dv, stats = _attn_bwd_args(q, k, v, out, dout, lse, scale,
                                                           dq, dk, dv, stats)
    _require(order, "order")
    if order.dtype != torch.int32 or order.numel() != N:
        raise HLAError(HLA_ERR_INVALID_ARG, f"order must be int32 with N = {N} entries")
    _check(lib().hla_attn_bwd_perm(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(lse),
                                   _ptr(order), ctypes.byref(mask.struct), _ptr(dq), _ptr(dk),
                                   _ptr(dv), _ptr(stats), B, Hh, N, d, _dtype_code(q), scale,
                                   _stream(q)))
    return dq, dk, dv


def attn_bwd_noalloc(q, k, v, out, dout, lse, mask: BlockMask, scale: Optional[float] = None,
                     dq: Optional[torch.Tensor] = None, dk: Optional[torch.Tensor] = None,
                     dv: Optional[torch.Tensor] = None):
    """hla_attn_bwd_noalloc: the backward with the row statistics in the library's own
    per-device array (B * heads * N <= 2^20) instead of a workspace. The library
    allocates nothing; pass dq, dk, dv to make the call allocate nothing here either.
    Calls that overlap in time on one device race. Returns (dq, dk, dv)."""
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (out, "out"), (dout, "dout"), (lse, "lse")):
        _require(t, n)
    if q.dim() != 4 or any(t.shape != q.shape for t in (k, v, out, dout)):
        raise HLAError(HLA_ERR_INVALID_ARG, "q, k, v, out, dout must all be [B, heads, N, d] of one shape")
    B, Hh, N, d = q.shape
    scale = 1.0 / float(d) ** 0.5 if scale is None else float(scale)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    for t, n in ((dq, "dq"), (dk, "dk"), (dv, "dv")):
        _require(t, n)
    _check(lib().hla_attn_bwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(lse),
                                      ctypes.byref(mask.struct), _ptr(dq), _ptr(dk), _ptr(dv),
                                      B, Hh, N, d, _dtype_code(q), scale, _stream(q)))
    return dq, dk, dv


def qkv_proj(x: torch.Tensor, w_qkv: torch.Tensor, heads: int, outs=None,
             order: Optional[torch.Tensor] = None):
    """x [B, N, C] -> q, k, v [B, heads, N, C/heads] (hla_qkv_proj).
    ``outs`` = preallocated (q, k, v) to write into. With ``order`` (int32 [N], the
    Hilbert order) x is in grid order and q, k, v come out in sequence order, the
    gather fused in (hla_qkv_proj_perm)."""
    _require(x, "x")
    _require(w_qkv, "w_qkv")
    if x.dtype != torch.bfloat16 or w_qkv.dtype != torch.bfloat16:
        raise HLAError(HLA_ERR_UNSUPPORTED, "qkv_proj takes bfloat16 x and w_qkv")
    B, N, C = x.shape
    d = C // heads
    if outs is None:
        outs = tuple(torch.empty((B, heads, N, d), dtype=x.dtype, device=x.device) for _ in range(3))
    q, k, v = outs
    if order is None:
        _check(lib().hla_qkv_proj(_ptr(x), _ptr(w_qkv), _ptr(q), _ptr(k), _ptr(v), B, N, heads, d,
                                  _stream(x)))
    else:
        _require_order(order, N)
        _check(lib().hla_qkv_proj_perm(_ptr(x), _ptr(w_qkv), _ptr(order), _ptr(q), _ptr(k), _ptr(v),
                                       B, N, heads, d, _stream(x)))
    return q, k, v


def out_proj(o: torch.Tensor, w_proj: torch.Tensor, out: Optional[torch.Tensor] = None,
             order: Optional[torch.Tensor] = None):
    """o [B, heads, N, d] -> y [B, N, C_out] (hla_out_proj). With ``order`` o is in
    sequence order and y comes out in grid order, the scatter fused in
    (hla_out_proj_perm)."""
    _require(o, "o")
    _require(w_proj, "w_proj")
    if o.dtype != torch.bfloat16 or w_proj.dtype != torch.bfloat16:
        raise HLAError(HLA_ERR_UNSUPPORTED, "out_proj takes bfloat16 o and w_proj")
    B, Hh, N, d = o.shape
    c_out = w_proj.shape[0]
    if out is None:
        out = torch.empty((B, N, c_out), dtype=o.dtype, device=o.device)
    if order is None:
        _check(lib().hla_out_proj(_ptr(o), _ptr(w_proj), _ptr(out), B, N, Hh, d, c_out, _stream(o)))
    else:
        _require_order(order, N)
        _check(lib().hla_out_proj_perm(_ptr(o), _ptr(w_proj), _ptr(order), _ptr(out), B, N, Hh, d,
                                       c_out, _stream(o)))
    return out
