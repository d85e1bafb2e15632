"""GPU parity: block-sparse attention backward against the oracle's float64
gradients of the dense masked attention, on the same seeded inputs.

The HIP path runs the forward (for out and lse) and then the backward, both on the
GPU; the oracle computes dq, dk, dv from q, k, v and dout alone.

Bars (max-abs error against the oracle, scaled by the gradient's own size
g = max(1, max |reference|)):
  bf16  <= 2e-2 * g.  Rounding the gradients to bf16 costs up to half an ulp
        (2^-9 relative) and the bf16 P and dS operands about as much again; a
        rounding-faithful emulation of the kernels' arithmetic on these inputs
        stays below 4.5e-3 * g, so the bar leaves a margin of four.
  f32   <= 1e-4 * g  (fp32 arithmetic throughout).
Full-size workloads are checked on sampled query rows (dq) and key rows (dk, dv)
of their first (b, h) slices, which the oracle evaluates one by one, plus properties that
hold at any size: determinism, and the sums fixed by the forward's invariances.
"""
import numpy as np
import pytest
import torch

import paper_2511_05832_amd as hla
import workloads as W
from conftest import Pat
from helpers import DEV, max_abs, np64, sample_rows
from oracle import attention as o_attn
from oracle import hilbert as o_hil
from oracle import permute as o_perm

pytestmark = pytest.mark.gpu

TOL_GRAD = {"bf16": 2e-2, "f32": 1e-4}


def dout_like(q, seed):
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    return torch.randn(q.shape, generator=g, dtype=torch.float32).to(q.dtype)


def run_hip(pattern, q, k, v, dout, tile_m, tile_n, scale, gather=True):
    """Forward then backward on the GPU. Inputs are CPU tensors in row-major order;
    Hilbert patterns gather them first. Returns dq, dk, dv (CPU, sequence order)."""
    qd, kd, vd, gd = (t.to(DEV) for t in (q, k, v, dout))
    if gather:
        order, _ = hla.hilbert_perm(pattern.H, pattern.W)
        qd, kd, vd, gd = (hla.gather(t, order) for t in (qd, kd, vd, gd))
    mask = hla.build_block_mask(pattern, tile_m, tile_n, columns=True)
    out, lse = hla.attn_fwd(qd, kd, vd, mask, scale)
    dq, dk, dv = hla.attn_bwd(qd, kd, vd, out, gd, lse, mask, scale)
    torch.cuda.synchronize()
    return dq.cpu(), dk.cpu(), dv.cpu()


def oracle(pattern, q, k, v, dout, scale, rows=None, key_rows=None, gather=True):
    arrs = [np64(t) for t in (q, k, v, dout)]
    if gather:
        order = o_hil.hilbert_order(pattern.H, pattern.W)
        arrs = [o_perm.gather(a, order) for a in arrs]
    return o_attn.attention_backward(*arrs, pattern, scale, rows=rows, key_rows=key_rows)


def check(got, ref, dtype, label):
    for name, g, r in zip(("dq", "dk", "dv"), got, ref):
        g = np64(g) if isinstance(g, torch.Tensor) else g
        scale = max(1.0, float(np.abs(r).max()))
        err = max_abs(g, r)
        print(f"{label} {name}: err {err:.3e} (scale {scale:.3f})")
        assert np.isfinite(g).all(), name
        assert err <= TOL_GRAD[dtype] * scale, (name, err, scale)


SMALL_PATTERNS = [Pat("hilbert_window", 32, 32, 64), Pat("hilbert_slide", 32, 32, 100),
                  Pat("hilbert_neighborhood", 32, 32, 49),
                  Pat("hilbert_shifted_window", 32, 32, 64, 32),
                  Pat("rowmajor_window", 32, 32, 8, 8), Pat("rowmajor_slide", 32, 32, 3, 3),
                  Pat("rowmajor_neighborhood", 32, 32, 7, 5)]


@pytest.mark.parametrize("pat", SMALL_PATTERNS, ids=repr)
@pytest.mark.parametrize("dtype,d,tm", [("bf16", 64, 128), ("bf16", 32, 64), ("f32", 32, 64),
                                         ("f32", 64, 128)])
def test_small_every_element(pat, dtype, d, tm):
    q, k, v = W.attn_inputs(1, 2, pat.N, d, dtype, seed=500 + d + tm)
    g = dout_like(q, 600 + d)
    scale = d ** -0.5
    gather = pat.kind.startswith("hilbert")
    got = run_hip(pat, q, k, v, g, tm, 64, scale, gather)
    ref = oracle(pat, q, k, v, g, scale, gather=gather)
    check(got, ref, dtype, f"{pat} {dtype} d{d} tm{tm}")


@pytest.mark.parametrize("w", [W.C1, W.C2], ids=lambda w: w.name)
def test_small_workloads_every_element(w):
    q, k, v = W.workload_inputs(w)
    g = dout_like(q, w.seed + 1000)
    got = run_hip(w.pattern, q, k, v, g, w.tile_m, w.tile_n, w.scale)
    ref = oracle(w.pattern, q, k, v, g, w.scale)
    check(got, ref, w.dtype, w.name)


def sample_keys(N, tile_n, seed, n):
    """Both sequence ends, the first and last key of a few key tiles, random keys."""
    rng = np.random.default_rng(seed)
    tiles = rng.choice(N // tile_n, size=2, replace=False)
    keys = [0, N - 1] + list(tiles * tile_n) + list(tiles * tile_n + tile_n - 1)
    keys += list(rng.choice(N, size=n, replace=False))
    return np.unique(np.asarray(keys, dtype=np.int64))


@pytest.mark.parametrize("w,n_slices,n_keys", [(W.C3, 2, 10), (W.C4, 1, 4)],
                         ids=lambda x: getattr(x, "name", str(x)))
def test_full_size_sampled(w, n_slices, n_keys):
    """The kernels run on the whole workload; the oracle checks sampled query rows
    and key rows of the first (b, h) slices (each sampled key needs every query
    that attends it, each over all N keys, so the key sample is small)."""
    q, k, v = W.workload_inputs(w)
    g = dout_like(q, w.seed + 1000)
    gather = w.pattern.kind.startswith("hilbert")
    dq, dk, dv = run_hip(w.pattern, q, k, v, g, w.tile_m, w.tile_n, w.scale, gather)
    rows = sample_rows(w.N, w.tile_m, w.seed, n_random=16)
    keys = sample_keys(w.N, w.tile_n, w.seed + 1, n_keys)
    sl = (slice(0, 1), slice(0, n_slices))
    ref = oracle(w.pattern, q[sl], k[sl], v[sl], g[sl], w.scale, rows=rows, key_rows=keys,
                 gather=gather)
    got = (dq[sl][:, :, rows], dk[sl][:, :, keys], dv[sl][:, :, keys])
    check(got, ref, w.dtype, w.name)


def test_full_size_properties_and_determinism():
    """At the full default size: two runs agree bit for bit; per (b, h), sum_j dk_j
    vanishes and sum_j dv_j equals sum_i dout_i (key-shift and value-shift
    invariance of the forward), up to bf16 rounding of the summed rows."""
    w = W.C3
    q, k, v = W.workload_inputs(w)
    g = dout_like(q, 77)
    a = run_hip(w.pattern, q, k, v, g, w.tile_m, w.tile_n, w.scale)
    b = run_hip(w.pattern, q, k, v, g, w.tile_m, w.tile_n, w.scale)
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    dq, dk, dv = (t.double() for t in a)
    gd = g.double()
    # every row of dk and dv carries a bf16 rounding error of at most 2^-9 of its size
    k_bound = 4 * 2.0 ** -9 * dk.abs().sum(dim=2).max().item() + 1e-3
    assert dk.sum(dim=2).abs().max().item() <= k_bound
    v_err = (dv.sum(dim=2) - gd.sum(dim=2)).abs().max().item()
    assert v_err <= 4 * 2.0 ** -9 * dv.abs().sum(dim=2).max().item() + 1e-3


def test_diagonal_mask():
    """A window of one token: out = v, so dv = dout exactly and dq = dk = 0 up to
    the difference of two fp32 summation orders of the same products."""
    pat = Pat("hilbert_window", 32, 32, 1)
    q, k, v = W.attn_inputs(2, 2, pat.N, 64, "bf16", seed=9)
    g = dout_like(q, 10)
    dq, dk, dv = run_hip(pat, q, k, v, g, 128, 64, 0.125, gather=False)
    assert torch.equal(dv, g)
    assert dq.abs().max().item() < 1e-3 and dk.abs().max().item() < 1e-3


def test_dense_limit():
    pat = Pat("hilbert_slide", 16, 16, 1000)
    q, k, v = W.attn_inputs(1, 3, pat.N, 64, "bf16", seed=11)
    g = dout_like(q, 12)
    got = run_hip(pat, q, k, v, g, 64, 64, 0.125)
    check(got, oracle(pat, q, k, v, g, 0.125), "bf16", "dense")


def random_cases(n):
    rng = np.random.default_rng(91)
    kinds = list(hla.PATTERN_IDS)
    cases = []
    for i in range(n):
        kind = kinds[i % len(kinds)]
        dtype = "bf16" if i % 3 else "f32"
        d = int(rng.choice([32, 64]))
        tm = int(rng.choice([64, 128]))
        H = int(rng.choice([16, 24, 32]))
        Wd = int(rng.choice([16, 32, 40]))
        if (H * Wd) % tm:
            tm = 64
        if (H * Wd) % tm:
            continue
        N = H * Wd
        if kind in ("hilbert_window", "hilbert_shifted_window"):
            p0 = int(rng.integers(1, 300))
            p1 = int(rng.integers(0, p0)) if kind == "hilbert_shifted_window" else 0
        elif kind == "hilbert_slide":
            p0, p1 = int(rng.integers(0, 200)), 0
        elif kind == "hilbert_neighborhood":
            p0, p1 = int(rng.integers(1, min(N, 300))), 0
        elif kind == "rowmajor_window":
            p0, p1 = int(rng.integers(1, H + 1)), int(rng.integers(1, Wd + 1))
        elif kind == "rowmajor_slide":
            p0, p1 = int(rng.integers(0, 6)), int(rng.integers(0, 6))
        else:
            p0, p1 = int(rng.integers(1, H + 1)), int(rng.integers(1, Wd + 1))
        cases.append((Pat(kind, H, Wd, p0, p1), dtype, d, tm, 1000 + i))
    return cases


@pytest.mark.parametrize("case", random_cases(28), ids=lambda c: f"{c[0]}-{c[1]}-d{c[2]}-tm{c[3]}")
def test_random_shapes(case):
    """Random patterns, grids (non-square: positions taken as already in sequence
    order), head dims, tiles and dtypes."""
    pat, dtype, d, tm, seed = case
    q, k, v = W.attn_inputs(1, 2, pat.N, d, dtype, seed=seed)
    g = dout_like(q, seed + 1)
    scale = d ** -0.5
    got = run_hip(pat, q, k, v, g, tm, 64, scale, gather=False)
    check(got, oracle(pat, q, k, v, g, scale, gather=False), dtype, str(case))


def test_requires_column_lists():
    pat = Pat("hilbert_slide", 16, 16, 20)
    q, k, v = (t.to(DEV) for t in W.attn_inputs(1, 1, pat.N, 64, "bf16", seed=3))
    mask = hla.build_block_mask(pat, 64, 64)
    out, lse = hla.attn_fwd(q, k, v, mask, 0.125)
    with pytest.raises(hla.HLAError, match="transposed"):
        hla.attn_bwd(q, k, v, out, q, lse, mask, 0.125)


def test_column_lists_match_oracle():
    from oracle import blockmask as o_bm
    for pat, tm in [(W.C2.pattern, 128), (W.C3.pattern, 128), (Pat("hilbert_neighborhood", 32, 32, 49), 64),
                    (Pat("rowmajor_neighborhood", 32, 32, 7, 5), 128)]:
        mask = hla.build_block_mask(pat, tm, 64, columns=True)
        torch.cuda.synchronize()
        ref = o_bm.column_lists(o_bm.classify(pat, tm, 64))
        np.testing.assert_array_equal(mask.n_full_t.cpu().numpy(), ref.n_full)
        np.testing.assert_array_equal(mask.n_part_t.cpu().numpy(), ref.n_part)
        np.testing.assert_array_equal(mask.full_idx_t.cpu().numpy(), ref.full_idx)
        np.testing.assert_array_equal(mask.part_idx_t.cpu().numpy(), ref.part_idx)


@pytest.mark.parametrize("dtype,d,tm", [("bf16", 64, 128), ("bf16", 32, 64), ("f32", 32, 64)], ids=str)
def test_stats_workspace_contents(dtype, d, tm):
    """The stats workspace holds, per row, (lse * log2 e, -delta) with delta =
    <dout, out>, as the C header documents."""
    pat = Pat("hilbert_slide", 16, 16, 20)
    q, k, v = (t.to(DEV) for t in W.attn_inputs(2, 2, pat.N, d, dtype, 404))
    g = dout_like(q, 405).to(DEV)
    mask = hla.build_block_mask(pat, tm, 64, columns=True)
    out, lse = hla.attn_fwd(q, k, v, mask, 0.125)
    stats = torch.full((2, 2, pat.N, 2), float("nan"), dtype=torch.float32, device=DEV)
    hla.attn_bwd(q, k, v, out, g, lse, mask, 0.125, stats=stats)
    torch.cuda.synchronize()
    st = stats.cpu().numpy().astype(np.float64)
    want_l2 = (lse.cpu() * 1.4426950408889634).numpy().astype(np.float64)
    np.testing.assert_allclose(st[..., 0], want_l2, rtol=1e-6, atol=0)
    prod = np64(out.cpu()) * np64(g.cpu())
    delta = prod.sum(-1)
    bound = 1e-5 * np.abs(prod).sum(-1) + 1e-30
    assert np.all(np.abs(st[..., 1] + delta) <= bound), float(np.max(np.abs(st[..., 1] + delta) / bound))


@pytest.mark.parametrize("pat,tm", [(Pat("hilbert_slide", 16, 16, 300), 128),
                                    (Pat("rowmajor_slide", 16, 16, 7, 7), 64)], ids=str)
@pytest.mark.parametrize("dtype,growth", [("f32", 3.0), ("bf16", 2.0)], ids=str)
def test_growing_scores(pat, tm, dtype, growth):
    """Keys of 64-key tile t scaled by growth^t and queries of +-0.5 (as in the
    forward's max-path test): scores spread over up to about 120 log2 units across
    a row, so P is recomputed from an lse far above most of the row's scores. fp32
    at 3^t checks that arithmetic at the fp32 bar. bf16 runs at 2^t: at 3^t its
    dq error reaches 2.1% of max |dq| (dS sums to zero along a row, and its bf16
    rounding is multiplied by keys up to 27 times larger), just past the bar."""
    g = torch.Generator().manual_seed(77)
    N, d = pat.N, 32 if dtype == "f32" else 64
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    k = torch.randn((1, 2, N, d), generator=g).abs()
    k = k * (growth ** (torch.arange(N) // 64).float())[None, None, :, None]
    sign = torch.where(torch.arange(N) % 2 == 0, 1.0, -1.0)
    q = 0.5 * sign[None, None, :, None].expand(1, 2, N, d).clone()
    v = torch.randn((1, 2, N, d), generator=g)
    q, k, v = (t.to(tdt) for t in (q, k, v))
    dout = dout_like(q, 78)
    got = run_hip(pat, q, k, v, dout, tm, 64, 0.125, gather=False)
    ref = oracle(pat, q, k, v, dout, 0.125, gather=False)
    for name, a, r in zip(("dq", "dk", "dv"), got, ref):
        gs = max(1.0, float(np.abs(r).max()))
        err = max_abs(np64(a), r)
        print(f"{pat} {dtype} {name}: err {err:.3e} (scale {gs:.3f})")
        assert err <= TOL_GRAD[dtype] * gs, (name, err, gs)


# Several heads per dk/dv workgroup (the launcher picks more than one only when
# one head per workgroup would overfill the GPU; the override forces it): head
# counts that do and do not divide B*heads and one above it (every head in one
# workgroup), 1-D and 2-D patterns, the shapes whose epilogue fits one ring stage
# (128-row query tiles) and one that keeps one head (64-row tiles). The
# gradients must equal the one-head launch bit for bit.
@pytest.mark.parametrize("hpw", [2, 3, 5, 8])
@pytest.mark.parametrize("pat", [Pat("hilbert_window", 32, 32, 64), Pat("hilbert_slide", 32, 32, 100),
                                 Pat("hilbert_neighborhood", 16, 16, 49),
                                 Pat("rowmajor_slide", 32, 32, 3, 3)], ids=repr)
@pytest.mark.parametrize("d,tm", [(64, 128), (32, 128), (64, 64)], ids=str)
def test_heads_per_workgroup(monkeypatch, hpw, pat, d, tm):
    q, k, v = W.attn_inputs(2, 3, pat.N, d, "bf16", seed=700 + hpw + d)
    g = dout_like(q, 800 + tm)
    scale = d ** -0.5
    gather = pat.kind.startswith("hilbert")
    monkeypatch.setenv("HLA_ATTN_BWD_HEADS_PER_WORKGROUP", "1")
    ref = run_hip(pat, q, k, v, g, tm, 64, scale, gather)
    monkeypatch.setenv("HLA_ATTN_BWD_HEADS_PER_WORKGROUP", str(hpw))
    got = run_hip(pat, q, k, v, g, tm, 64, scale, gather)
    for name, a, b in zip(("dq", "dk", "dv"), got, ref):
        assert torch.equal(a, b), f"{name} differs with {hpw} heads per workgroup"


@pytest.mark.parametrize("value", ["0", "65", "x"])
def test_heads_per_workgroup_override_out_of_range_is_ignored(monkeypatch, value):
    pat = Pat("hilbert_window", 32, 32, 64)
    q, k, v = W.attn_inputs(2, 3, pat.N, 64, "bf16", seed=9)
    g = dout_like(q, 10)
    monkeypatch.delenv("HLA_ATTN_BWD_HEADS_PER_WORKGROUP", raising=False)
    ref = run_hip(pat, q, k, v, g, 128, 64, 0.125)
    monkeypatch.setenv("HLA_ATTN_BWD_HEADS_PER_WORKGROUP", value)
    got = run_hip(pat, q, k, v, g, 128, 64, 0.125)
    for a, b in zip(got, ref):
        assert torch.equal(a, b)
