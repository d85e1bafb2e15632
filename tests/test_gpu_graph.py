"""The whole hot path can be captured into a HIP graph and replayed: every replay,
with the program's own eager work and synchronisations in between, reproduces the
eager result bit for bit (the library enqueues no allocation, memset or host
synchronisation)."""
import pytest
import torch

import paper_2511_05832_amd as hla
import workloads as W

pytestmark = pytest.mark.gpu


def test_attention_step_graph_replays_match_eager():
    pat = W.Pattern(W.HILBERT_SLIDE, 32, 32, 100)
    B, Hh, N, d = 2, 2, 1024, 64
    q, k, v = (t.cuda() for t in W.attn_inputs(B, Hh, N, d, "bf16", seed=21))
    qh, kh, vh, oh, o = (torch.empty_like(q) for _ in range(5))
    lse = torch.empty((B, Hh, N), dtype=torch.float32, device="cuda")
    order = torch.empty(N, dtype=torch.int32, device="cuda")
    rank = torch.empty(N, dtype=torch.int32, device="cuda")
    mask = hla.BlockMask(pat, 128, 64)

    def step():
        hla.hilbert_perm(32, 32, out=(order, rank))
        for src, dst in ((q, qh), (k, kh), (v, vh)):
            hla.gather(src, order, out=dst)
        mask.build()
        hla.attn_fwd(qh, kh, vh, mask, 0.125, out=oh, lse=lse)
        hla.scatter(oh, order, out=o)

    step()
    torch.cuda.synchronize()
    ref_o, ref_lse, ref_lists = o.clone(), lse.clone(), mask.part_idx.clone()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for r in range(4):
        # eager work between replays that overwrites every intermediate
        for t in (qh, kh, vh, oh, o):
            t.normal_()
        lse.fill_(float("nan"))
        order.fill_(0)
        mask.part_idx.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o, ref_o), r
        assert torch.equal(lse, ref_lse), r
        assert torch.equal(mask.part_idx, ref_lists), r


def test_fused_attention_step_graph_replays_match_eager():
    """The measured step: the Hilbert index and the tile lists in one launch, then the
    attention with the reordering fused in, on grid-ordered q, k, v."""
    pat = W.Pattern(W.HILBERT_WINDOW, 64, 64, 256)
    B, Hh, N, d = 2, 2, 4096, 64
    q, k, v = (t.cuda() for t in W.attn_inputs(B, Hh, N, d, "bf16", seed=22))
    o = torch.empty_like(q)
    lse = torch.empty((B, Hh, N), dtype=torch.float32, device="cuda")
    order = torch.empty(N, dtype=torch.int32, device="cuda")
    rank = torch.empty(N, dtype=torch.int32, device="cuda")
    mask = hla.BlockMask(pat, 128, 64, totals=False)

    def step():
        mask.build_with_path(order, rank)
        hla.attn_fwd_perm(q, k, v, order, mask, 0.125, out=o, lse=lse)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (o, lse, order, rank, mask.full_idx, mask.n_full)]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for r in range(4):
        o.normal_()
        lse.fill_(float("nan"))
        order.fill_(0)
        rank.fill_(-1)
        mask.full_idx.fill_(-7)
        mask.n_full.fill_(3)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for got, want in zip((o, lse, order, rank, mask.full_idx, mask.n_full), ref):
            assert torch.equal(got, want), r


def test_layer_step_graph_replays_match_eager():
    w = W.LayerWorkload("graph_layer", H=16, W=16, B=2, heads=2, d=32, half_width=20,
                        tile_m=128, tile_n=64, seed=22)
    x, wq, wp = (t.cuda() for t in W.layer_inputs(w))
    xh = torch.empty_like(x)
    qkv = [torch.empty((w.B, w.heads, w.N, w.d), dtype=torch.bfloat16, device="cuda") for _ in range(4)]
    yh, y = torch.empty_like(x), torch.empty_like(x)
    order = torch.empty(w.N, dtype=torch.int32, device="cuda")
    rank = torch.empty(w.N, dtype=torch.int32, device="cuda")
    mask = hla.BlockMask(w.pattern, w.tile_m, w.tile_n)

    def step():
        hla.hilbert_perm(w.H, w.W, out=(order, rank))
        hla.gather(x, order, out=xh)
        hla.qkv_proj(xh, wq, w.heads, outs=tuple(qkv[:3]))
        mask.build()
        hla.attn_fwd(qkv[0], qkv[1], qkv[2], mask, w.scale, out=qkv[3], with_lse=False)
        hla.out_proj(qkv[3], wp, out=yh)
        hla.scatter(yh, order, out=y)

    step()
    torch.cuda.synchronize()
    ref = y.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for r in range(3):
        for t in [xh, yh, y] + qkv:
            t.normal_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref), r


def test_backward_step_graph_replays_match_eager():
    pat = W.Pattern(W.HILBERT_WINDOW, 32, 32, 64)
    B, Hh, N, d = 2, 2, 1024, 64
    q, k, v = (t.cuda() for t in W.attn_inputs(B, Hh, N, d, "bf16", seed=23))
    g = torch.randn((B, Hh, N, d), generator=torch.Generator().manual_seed(24)).to(torch.bfloat16).cuda()
    mask = hla.BlockMask(pat, 128, 64, columns=True)
    out = torch.empty_like(q)
    lse = torch.empty((B, Hh, N), dtype=torch.float32, device="cuda")
    grads = [torch.empty_like(q) for _ in range(3)]
    stats = torch.empty((B, Hh, N, 2), dtype=torch.float32, device="cuda")

    def step():
        mask.build()
        hla.attn_fwd(q, k, v, mask, 0.125, out=out, lse=lse)
        hla.attn_bwd(q, k, v, out, g, lse, mask, 0.125, dq=grads[0], dk=grads[1], dv=grads[2],
                     stats=stats)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in grads]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for r in range(3):
        for t in grads + [out]:
            t.normal_()
        stats.fill_(float("nan"))
        mask.part_idx_t.fill_(-3)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for a, b in zip(grads, ref):
            assert torch.equal(a, b), r
