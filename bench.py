"""Benchmark of the Hilbert-guided block-sparse attention hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--all]

A step is one pass of the whole hot path over one batch of synthetic input
already resident in HBM: Hilbert index and inverse, gather of q, k, v into
Hilbert order, tile classification and lists, block-sparse attention forward,
scatter of the output back to row-major (for the layer workload: gather of the
features, QKV projection, attention, output projection, scatter). Input buffer
sets are rotated from step to step so that the working set exceeds the 256 MB
Infinity Cache and every step reads from HBM.

Prints ONE JSON line on stdout. Timing uses HIP events on the stream every
kernel is launched on (torch's current stream): one pair around the K timed
steps, and one pair around every launch of each stage, which gives each
kernel's average duration inside the timed region. The default workload is the
128x128-token Hilbert window attention (B=4, heads=8, d=64, window 256), the
same batch x heads x tokens x head_dim as the paper's headline window row
(Table 1, I=128x128, W=16x16). The same kernel is then timed on the row-major
16x16 window mask for the empty-tile comparison, and the CPU oracle is timed
on a bounded sample of the same step on the host cores.

The backward pass of the same attention workload is timed the same way (a
graph-replayed step: gather of the upstream gradient, hla_attn_bwd, scatter of
dq, dk, dv; per-call time of hla_attn_bwd from an eager pass) and reported under
"backward"; with the reordering fused in (hla_attn_bwd_perm on the grid-ordered
tensors) under "backward_fused"; --no-backward skips both. The attention with the global relative
position bias (hla_attn_fwd_rpb) is timed per call on the same inputs and
reported under "rpb"; --no-rpb skips it.

Every measured configuration (the 32x32 fp32 window, the 64x64 and 256x256
bands, the 128x128 window, the row-major twins run through the same kernel, and
the 64x64 layer) then gets a record under "configs": its step, its attention
kernel alone (back-to-back launches) with TFLOP/s, % of its dtype's peak and a
roofline record, and, for the Hilbert ones, the gather and scatter kernels with
GB/s and the fraction of the 8 TB/s HBM peak. The Hilbert index is timed at
128x128, 256x256 and 4096x4096 under "hilbert_index". --no-configs skips both.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import platform
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import torch  # noqa: E402

import workloads as W  # noqa: E402

METRIC = "attn fwd ms/call + TFLOP/s on non-empty tiles (% bf16 MFMA peak); perm GB/s"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3       # MI355X fp32 (vector and matrix)
MALL_BYTES = 256 << 20


def esize(dtype: str) -> int:
    return 2 if dtype == "bf16" else 4


def tdtype(dtype: str):
    return torch.bfloat16 if dtype == "bf16" else torch.float32


class Timer:
    """Per-stage event pairs on the current stream, averaged over the timed steps."""

    def __init__(self):
        self.pairs = {}
        self.active = False

    def stage(self, name):
        timer = self

        class _Ctx:
            def __enter__(self_inner):
                if timer.active:
                    self_inner.a = torch.cuda.Event(enable_timing=True)
                    self_inner.a.record()

            def __exit__(self_inner, *exc):
                if timer.active:
                    b = torch.cuda.Event(enable_timing=True)
                    b.record()
                    timer.pairs.setdefault(name, []).append((self_inner.a, b))
                return False
        return _Ctx()

    def mean_ms(self, name):
        ps = self.pairs.get(name, [])
        return sum(a.elapsed_time(b) for a, b in ps) / len(ps) if ps else float("nan")

    def median_ms(self, name):
        ts = sorted(a.elapsed_time(b) for a, b in self.pairs.get(name, []))
        return ts[len(ts) // 2] if ts else float("nan")

    def count(self, name):
        return len(self.pairs.get(name, []))


def b2b_ms(call, n):
    """Average duration of call(i) for n back-to-back launches between one event pair
    on the current stream (no event between launches); call(0) runs once before."""
    call(0)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(n):
        call(i + 1)
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / n


def roofline_record(kernel, ms, nbytes, flops, dtype):
    """The roofline of one kernel: HBM-bound when its algorithmic bytes take longer at
    the HBM peak than its FLOPs at the compute peak of its dtype, else compute-bound."""
    peak_tf = BF16_PEAK_TFLOPS if dtype == "bf16" else FP32_PEAK_TFLOPS
    t = ms * 1e-3
    rec = {"kernel": kernel, "kernel_ms_per_launch": ms, "algorithmic_bytes": nbytes,
           "algorithmic_flops": flops}
    if nbytes / (HBM_PEAK_GBS * 1e9) >= flops / (peak_tf * 1e12):
        ach = nbytes / t / 1e9
        rec.update(bound="hbm", achieved=ach, peak=HBM_PEAK_GBS, unit="GB/s", frac=ach / HBM_PEAK_GBS,
                   compute_frac=(flops / t / 1e12) / peak_tf if flops else 0.0)
    else:
        ach = flops / t / 1e12
        rec.update(bound="mfma" if dtype == "bf16" else "fp32", achieved=ach, peak=peak_tf,
                   unit="TFLOP/s", frac=ach / peak_tf, hbm_frac=nbytes / t / 1e9 / HBM_PEAK_GBS)
    return rec


def perm_record(kernel_ms, nbytes, traffic=None):
    """A permutation kernel: algorithmic bytes (tensor read and written once, plus
    the order array) per launch, their rate, its fraction of the HBM peak, and the
    counter-measured bytes per launch where a current summary exists."""
    gbs = nbytes / (kernel_ms * 1e-3) / 1e9
    return {"ms_per_call": kernel_ms, "gbs": gbs, "frac": gbs / HBM_PEAK_GBS, "bytes": nbytes,
            "traffic": traffic}


# ----------------------------------------------------------------------------
# attention workloads


def single_ok(w) -> bool:
    """hla_attn_fwd_hilbert covers the workload: a 1-D Hilbert pattern on a 2^k x 2^k
    grid (side >= 8), bf16."""
    p = getattr(w, "pattern", None)
    return (p is not None and p.hilbert and getattr(w, "dtype", "bf16") == "bf16" and p.H == p.W
            and p.W >= 8 and (p.W & (p.W - 1)) == 0)


class AttnPipeline:
    """One step of an attention workload. Hilbert patterns either reorder with
    separate gather and scatter passes around hla_attn_fwd (composed), or hand the
    grid-ordered tensors and the Hilbert order to hla_attn_fwd_perm, which does the
    reordering inside its loads and stores (fused), or run the whole step - index,
    tile lists, reordered attention - as one launch of hla_attn_fwd_hilbert
    (single)."""

    def __init__(self, w: W.AttnWorkload, hla, fused: bool = False, single: bool = False):
        self.w, self.hla = w, hla
        pat = w.pattern
        self.hilbert = pat.hilbert
        self.single = single and single_ok(w)
        self.fused = (fused or self.single) and self.hilbert
        B, Hh, N, d = w.B, w.heads, w.N, w.d
        tensor_bytes = B * Hh * N * d * esize(w.dtype)
        set_bytes = tensor_bytes * (7 if self.hilbert and not self.fused else 4)
        self.nsets = max(2, min(64, math.ceil(3 * MALL_BYTES / set_bytes)))
        q, k, v = W.workload_inputs(w)
        self.sets = []
        for i in range(self.nsets):
            s = {"q": q.cuda(), "k": k.cuda(), "v": v.cuda()}
            if self.hilbert and not self.fused:
                for n in ("qh", "kh", "vh", "oh"):
                    s[n] = torch.empty_like(s["q"])
            s["o"] = torch.empty_like(s["q"])
            s["lse"] = torch.empty((B, Hh, N), dtype=torch.float32, device="cuda")
            self.sets.append(s)
        del q, k, v
        self.order = torch.empty(N, dtype=torch.int32, device="cuda")
        self.rank = torch.empty(N, dtype=torch.int32, device="cuda")
        self.mask = hla.BlockMask(pat, w.tile_m, w.tile_n, totals=False)
        if self.single:
            # the step computes its own; these serve the FLOP count and the backward
            self.mask.build_with_path(self.order, self.rank)
        self.timer = Timer()

    def step(self, i):
        hla, w, s, T = self.hla, self.w, self.sets[i % self.nsets], self.timer
        if self.single:
            with T.stage("attn"):
                hla.attn_fwd_hilbert(s["q"], s["k"], s["v"], w.pattern, w.tile_m, w.tile_n, w.scale,
                                     out=s["o"], lse=s["lse"])
            return
        if self.fused:
            with T.stage("path_mask"):
                self.mask.build_with_path(self.order, self.rank)
            with T.stage("attn"):
                hla.attn_fwd_perm(s["q"], s["k"], s["v"], self.order, self.mask, w.scale,
                                  out=s["o"], lse=s["lse"])
            return
        if self.hilbert:
            with T.stage("path_mask"):
                self.mask.build_with_path(self.order, self.rank)
            with T.stage("gather"):
                for a, b in (("q", "qh"), ("k", "kh"), ("v", "vh")):
                    hla.gather(s[a], self.order, out=s[b])
            qn, kn, vn, on = "qh", "kh", "vh", "oh"
        else:
            qn, kn, vn, on = "q", "k", "v", "o"
            with T.stage("mask"):
                self.mask.build()
        with T.stage("attn"):
            hla.attn_fwd(s[qn], s[kn], s[vn], self.mask, w.scale, out=s[on], lse=s["lse"])
        if self.hilbert:
            with T.stage("scatter"):
                hla.scatter(s["oh"], self.order, out=s["o"])

    def kernel_ms(self, n):
        """Average duration of the attention kernel alone: n back-to-back launches
        (rotating input sets, the step's order and tile lists) between one event pair
        on the stream they are launched on, so no per-launch event sits between them."""
        hla, w = self.hla, self.w

        def call(i):
            s = self.sets[i % self.nsets]
            if self.single:
                hla.attn_fwd_hilbert(s["q"], s["k"], s["v"], w.pattern, w.tile_m, w.tile_n, w.scale,
                                     out=s["o"], lse=s["lse"])
            elif self.fused:
                hla.attn_fwd_perm(s["q"], s["k"], s["v"], self.order, self.mask, w.scale,
                                  out=s["o"], lse=s["lse"])
            else:
                qn, kn, vn, on = ("qh", "kh", "vh", "oh") if self.hilbert else ("q", "k", "v", "o")
                hla.attn_fwd(s[qn], s[kn], s[vn], self.mask, w.scale, out=s[on], lse=s["lse"])
        call(0)
        torch.cuda.synchronize()
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        for i in range(n):
            call(i + 1)
        end.record()
        torch.cuda.synchronize()
        return start.elapsed_time(end) / n

    def perm_kernel_ms(self, n, scatter=False):
        """Average duration of one gather (or scatter) of a [B, heads, N, d] tensor:
        n back-to-back launches on rotating input sets between one event pair."""
        hla = self.hla
        if scatter:
            return b2b_ms(lambda i: hla.scatter(self.sets[i % self.nsets]["oh"], self.order,
                                                out=self.sets[i % self.nsets]["o"]), n)
        return b2b_ms(lambda i: hla.gather(self.sets[i % self.nsets]["q"], self.order,
                                           out=self.sets[i % self.nsets]["qh"]), n)

    # algorithmic figures -------------------------------------------------
    def tile_flops(self):
        tf, tp = self.mask.host_totals()
        w = self.w
        return 4.0 * w.tile_m * w.tile_n * w.d * (tf + tp) * w.B * w.heads, tf, tp

    def attn_bytes(self):
        """q, k, v, out once each plus the fp32 log-sum-exp: 4 N d s + 4 N per (b, h)."""
        w = self.w
        return (4 * w.N * w.d * esize(w.dtype) + 4 * w.N) * w.B * w.heads

    def perm_bytes_per_tensor(self):
        """One gather or scatter of a [B, heads, N, d] tensor: read + write + int32 index."""
        w = self.w
        return 2 * w.B * w.heads * w.N * w.d * esize(w.dtype) + 4 * w.N


    # backward ------------------------------------------------------------
    def setup_backward(self):
        """Buffers of the backward pass for every input set (after the forward has run
        on every set, so out and lse are valid): an upstream gradient in row-major
        order and the gradients; the mask with its per-column lists."""
        hla, w = self.hla, self.w
        g = torch.Generator(device="cpu")
        g.manual_seed(w.seed + 1000)
        dout = torch.randn((w.B, w.heads, w.N, w.d), generator=g).to(tdtype(w.dtype))
        for s in self.sets:
            s["dout"] = dout.cuda()
            for n in ("dq", "dk", "dv"):
                s[n] = torch.empty_like(s["q"])
            if self.hilbert and not self.fused:
                s["douth"] = torch.empty_like(s["q"])
                for n in ("dqr", "dkr", "dvr"):
                    s[n] = torch.empty_like(s["q"])
            s["stats"] = torch.empty((w.B, w.heads, w.N, 2), dtype=torch.float32, device="cuda")
        self.mask_c = hla.BlockMask(w.pattern, w.tile_m, w.tile_n, columns=True).build()
        self.timer_bwd = Timer()

    def step_backward(self, i):
        """Gather the upstream gradient into the forward's order, run the backward,
        scatter dq, dk, dv back to row-major (fused: hla_attn_bwd_perm on the
        grid-ordered tensors, no gather or scatter)."""
        hla, w, s, T = self.hla, self.w, self.sets[i % self.nsets], self.timer_bwd
        if self.fused:
            with T.stage("attn_bwd"):
                hla.attn_bwd_perm(s["q"], s["k"], s["v"], s["o"], s["dout"], s["lse"], self.order,
                                  self.mask_c, w.scale, dq=s["dq"], dk=s["dk"], dv=s["dv"],
                                  stats=s["stats"])
            return
        if self.hilbert:
            with T.stage("gather"):
                hla.gather(s["dout"], self.order, out=s["douth"])
            names = ("qh", "kh", "vh", "oh", "douth")
        else:
            names = ("q", "k", "v", "o", "dout")
        with T.stage("attn_bwd"):
            hla.attn_bwd(*(s[n] for n in names), s["lse"], self.mask_c, w.scale,
                         dq=s["dq"], dk=s["dk"], dv=s["dv"], stats=s["stats"])
        if self.hilbert:
            with T.stage("scatter"):
                for a, b in (("dq", "dqr"), ("dk", "dkr"), ("dv", "dvr")):
                    hla.scatter(s[a], self.order, out=s[b])

    def bwd_bytes(self):
        """Algorithmic HBM bytes of one backward call: q, k, v, out, dout read and dq,
        dk, dv written once (8 N d s), lse read (4 N), row stats written and read
        (16 N), per (b, h)."""
        w = self.w
        return (8 * w.N * w.d * esize(w.dtype) + 20 * w.N) * w.B * w.heads

# ----------------------------------------------------------------------------
# layer workload


class LayerPipeline:
    """The layer step. single: the projections work in grid order (hla_qkv_proj,
    hla_out_proj) around the one-launch attention (hla_attn_fwd_hilbert, which
    takes its rows from the curve and classifies its tiles itself) - three
    launches, no index or list in memory. fused: the index and lists in one
    launch, the QKV projection reading x through the Hilbert order and the output
    projection writing y through it (hla_qkv_proj_perm, hla_out_proj_perm), the
    attention in sequence order. Otherwise separate gather and scatter passes
    around hla_qkv_proj and hla_out_proj."""

    def __init__(self, w: W.LayerWorkload, hla, fused: bool = True, single: bool = False):
        self.w, self.hla = w, hla
        self.single = single and single_ok(w)
        self.fused = fused and not self.single
        self.hilbert = True
        B, N, C, Hh, d = w.B, w.N, w.C, w.heads, w.d
        x, wq, wp = W.layer_inputs(w)
        set_bytes = B * N * C * 2 * 7
        self.nsets = max(2, min(64, math.ceil(3 * MALL_BYTES / set_bytes)))
        self.wq, self.wp = wq.cuda(), wp.cuda()
        self.sets = []
        for i in range(self.nsets):
            s = {"x": x.cuda()}
            s["xh"] = torch.empty_like(s["x"])
            for n in ("q", "k", "v", "o"):
                s[n] = torch.empty((B, Hh, N, d), dtype=torch.bfloat16, device="cuda")
            s["yh"] = torch.empty((B, N, C), dtype=torch.bfloat16, device="cuda")
            s["y"] = torch.empty_like(s["yh"])
            self.sets.append(s)
        self.order = torch.empty(N, dtype=torch.int32, device="cuda")
        self.rank = torch.empty(N, dtype=torch.int32, device="cuda")
        self.mask = hla.BlockMask(w.pattern, w.tile_m, w.tile_n, totals=False)
        if self.single:
            # the step computes its own; these serve the FLOP count
            self.mask.build_with_path(self.order, self.rank)
        self.timer = Timer()

    def step(self, i):
        hla, w, s, T = self.hla, self.w, self.sets[i % self.nsets], self.timer
        if self.single:
            with T.stage("qkv"):
                hla.qkv_proj(s["x"], self.wq, w.heads, outs=(s["q"], s["k"], s["v"]))
            with T.stage("attn"):
                hla.attn_fwd_hilbert(s["q"], s["k"], s["v"], w.pattern, w.tile_m, w.tile_n, w.scale,
                                     out=s["o"], with_lse=False)
            with T.stage("proj"):
                hla.out_proj(s["o"], self.wp, out=s["y"])
            return
        with T.stage("path_mask"):
            self.mask.build_with_path(self.order, self.rank)
        if self.fused:
            with T.stage("qkv"):
                hla.qkv_proj(s["x"], self.wq, w.heads, outs=(s["q"], s["k"], s["v"]), order=self.order)
            with T.stage("attn"):
                hla.attn_fwd(s["q"], s["k"], s["v"], self.mask, w.scale, out=s["o"], with_lse=False)
            with T.stage("proj"):
                hla.out_proj(s["o"], self.wp, out=s["y"], order=self.order)
            return
        with T.stage("gather"):
            hla.gather(s["x"], self.order, out=s["xh"])
        with T.stage("qkv"):
            hla.qkv_proj(s["xh"], self.wq, w.heads, outs=(s["q"], s["k"], s["v"]))
        with T.stage("attn"):
            hla.attn_fwd(s["q"], s["k"], s["v"], self.mask, w.scale, out=s["o"], with_lse=False)
        with T.stage("proj"):
            hla.out_proj(s["o"], self.wp, out=s["yh"])
        with T.stage("scatter"):
            hla.scatter(s["yh"], self.order, out=s["y"])

    def kernel_ms(self, which, n):
        """Average duration of one stage's kernel alone (qkv, attn, proj, gather,
        scatter), n back-to-back launches on rotating input sets; the projections
        take the step's order (fused) or none."""
        hla, w = self.hla, self.w
        order = self.order if self.fused else None

        def S(i):
            return self.sets[i % self.nsets]

        def attn(i):
            if self.single:
                hla.attn_fwd_hilbert(S(i)["q"], S(i)["k"], S(i)["v"], w.pattern, w.tile_m, w.tile_n, w.scale,
                                     out=S(i)["o"], with_lse=False)
            else:
                hla.attn_fwd(S(i)["q"], S(i)["k"], S(i)["v"], self.mask, w.scale, out=S(i)["o"], with_lse=False)
        calls = {
            "qkv": lambda i: hla.qkv_proj(S(i)["x"], self.wq, w.heads, outs=(S(i)["q"], S(i)["k"], S(i)["v"]),
                                          order=order),
            "attn": attn,
            "proj": lambda i: hla.out_proj(S(i)["o"], self.wp, out=S(i)["y"], order=order),
            "gather": lambda i: hla.gather(S(i)["x"], self.order, out=S(i)["xh"]),
            "scatter": lambda i: hla.scatter(S(i)["yh"], self.order, out=S(i)["y"]),
        }
        return b2b_ms(calls[which], n)

    def tile_flops(self):
        tf, tp = self.mask.host_totals()
        w = self.w
        return 4.0 * w.tile_m * w.tile_n * w.d * (tf + tp) * w.B * w.heads, tf, tp

    def attn_bytes(self):
        w = self.w
        return 4 * w.N * w.d * 2 * w.B * w.heads

    def proj_figures(self, which):
        """(algorithmic bytes, FLOPs) of one projection call: the activations read and
        written once, the weights once, the order array once when fused."""
        w = self.w
        T, C = w.B * w.N, w.C
        idx = 4 * w.N if self.fused else 0
        if which == "qkv":
            return 2 * (T * C + 3 * T * C + 3 * C * C) + idx, 2.0 * T * C * 3 * C
        return 2 * (T * C + T * C + C * C) + idx, 2.0 * T * C * C

    def perm_bytes_per_tensor(self):
        w = self.w
        return 2 * w.B * w.N * w.C * 2 + 4 * w.N


ATTN_SOURCES = ("paper_2511_05832_amd/csrc/attn_bf16.hip", "paper_2511_05832_amd/csrc/attn_common.h",
                "paper_2511_05832_amd/csrc/hla_internal.h", "paper_2511_05832_amd/csrc/hilbert_common.h",
                "paper_2511_05832_amd/csrc/tiles_common.h")
PERM_SOURCES = ("paper_2511_05832_amd/csrc/permute.hip", "paper_2511_05832_amd/csrc/hla_internal.h")
PROJ_SOURCES = ("paper_2511_05832_amd/csrc/proj.hip", "paper_2511_05832_amd/csrc/attn_common.h",
                "paper_2511_05832_amd/csrc/hla_internal.h")


def profile_traffic(name, sources):
    """HBM bytes per dispatch from the committed rocprofv3 counter summary
    profiles/<name>_traffic.txt, or None if there is none or one of the kernel's
    source files changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{name}_traffic.txt")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        k, sep, v = line.partition(":")
        if sep:
            fields[k.strip()] = v.strip()
    h = hashlib.sha256()
    for src in sources:
        h.update(open(os.path.join(ROOT, src), "rb").read())
    if fields.get("kernel_source_sha256") != h.hexdigest():
        return None
    try:
        return int(fields["traffic_bytes_per_dispatch"])
    except (KeyError, ValueError):
        return None


def measured_traffic(workload_name, kernel="attn_fwd"):
    """HBM bytes per attention dispatch (kernel attn_fwd, attn_fwd_perm or
    attn_fwd_rpb) on this workload from the committed counter summary."""
    return profile_traffic(f"{kernel}_bf16_{workload_name}", ATTN_SOURCES)


def make_pipeline(w, hla, fused=False, single=False):
    """A layer workload gets its default step: one launch for the attention where
    the pattern allows it, else the reordering fused into the projections."""
    return (LayerPipeline(w, hla, single=True) if isinstance(w, W.LayerWorkload)
            else AttnPipeline(w, hla, fused, single))


def capture_step_graphs(pipe):
    """One HIP graph per input set, each holding one whole step (every launch of the
    hot path on the capture stream; nothing in it allocates or memsets)."""
    graphs = []
    for i in range(pipe.nsets):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            pipe.step(i)
        graphs.append(g)
    torch.cuda.synchronize()
    return graphs


WARM_MS = 150.0


def warm_replays(graphs, warmup):
    """Untimed replays before a timed pass: the W warm-up steps, then more until
    WARM_MS of them have run, so the timed steps start at the GPU's steady clock
    (right after a pipeline is built the first ~5 ms of steps run up to 15%
    slower)."""
    for i in range(max(warmup, 1)):
        graphs[i % len(graphs)].replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    i = 0
    while (time.perf_counter() - t0) * 1e3 < WARM_MS:
        for _ in range(16):
            graphs[i % len(graphs)].replay()
            i += 1
        torch.cuda.synchronize()


def run_timed(pipe, steps, warmup):
    """Returns (ms per step, ms per step of the eager pass, {"graph": ms, "stream": ms}).

    The eager pass records one event pair around every stage, which gives each
    kernel's average duration. The K steps are then timed twice: replaying the
    captured graphs (no host launch gaps), and launched back to back from the host
    with no event between steps (a one-launch step then pays no graph-launch cost,
    about 5 us per replay). The step time is the faster of the two."""
    for i in range(warmup):
        pipe.step(i)
    torch.cuda.synchronize()
    pipe.timer.active = True
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    marks[0].record()
    for i in range(steps):
        pipe.step(warmup + i)
        marks[i + 1].record()
    torch.cuda.synchronize()
    pipe.timer.active = False
    # median step: a host stall of the eager loop (up to milliseconds, now and
    # then) would dominate the mean of a ~0.1 ms step
    eager_ms = statistics.median(marks[i].elapsed_time(marks[i + 1]) for i in range(steps))
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    graphs = capture_step_graphs(pipe)
    warm_replays(graphs, warmup)
    start.record()
    for i in range(steps):
        graphs[i % len(graphs)].replay()
    end.record()
    torch.cuda.synchronize()
    graph_ms = start.elapsed_time(end) / steps
    del graphs
    for i in range(max(warmup, 1)):
        pipe.step(i)
    torch.cuda.synchronize()
    start.record()
    for i in range(steps):
        pipe.step(warmup + i)
    end.record()
    torch.cuda.synchronize()
    stream_ms = start.elapsed_time(end) / steps
    return min(graph_ms, stream_ms), eager_ms, {"graph": graph_ms, "stream": stream_ms}


def time_backward(pipe, steps, warmup):
    """Backward pass of an attention workload: eager pass with stage events, then
    replays of one captured graph per input set (as for the forward)."""
    pipe.setup_backward()
    for i in range(warmup):
        pipe.step_backward(i)
    torch.cuda.synchronize()
    T = pipe.timer_bwd
    T.active = True
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(steps):
        pipe.step_backward(i)
    end.record()
    torch.cuda.synchronize()
    T.active = False
    eager_ms = start.elapsed_time(end) / steps
    graphs = []
    for i in range(pipe.nsets):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            pipe.step_backward(i)
        graphs.append(g)
    torch.cuda.synchronize()
    warm_replays(graphs, warmup)
    start.record()
    for i in range(steps):
        graphs[i % len(graphs)].replay()
    end.record()
    torch.cuda.synchronize()
    graph_ms = start.elapsed_time(end) / steps
    del graphs
    w = pipe.w
    tf, tp = pipe.mask.host_totals()
    tiles = (tf + tp) * w.B * w.heads
    # five products per non-empty tile (S, dP, dV, dK, dQ), the usual count; the
    # kernels recompute S and dP once more (seven products executed)
    flops = 10.0 * w.tile_m * w.tile_n * w.d * tiles
    # median per call: host stalls of the eager loop (up to milliseconds on some
    # boxes) land inside whichever event bracket is open and would skew a mean
    bwd_ms = T.median_ms("attn_bwd")
    peak = BF16_PEAK_TFLOPS if w.dtype == "bf16" else FP32_PEAK_TFLOPS
    tflops = flops / (bwd_ms * 1e-3) / 1e12
    return {
        "ms_per_step": graph_ms,
        "ms_per_step_eager": eager_ms,
        "step": ("attention backward with the reordering fused in (hla_attn_bwd_perm)" if pipe.fused
                 else "gather of dout, attention backward, scatter of dq, dk, dv" if pipe.hilbert
                 else "attention backward"),
        "attn_bwd_ms_per_call": bwd_ms,
        "attn_bwd_ms_per_call_mean": T.mean_ms("attn_bwd"),
        "tile_flops": flops,
        "tile_flops_executed": 1.4 * flops,
        "attn_bwd_tflops_nonempty_tiles": tflops,
        "attn_bwd_pct_peak": 100.0 * tflops / peak,
        "attn_bwd_algorithmic_gbs": pipe.bwd_bytes() / (bwd_ms * 1e-3) / 1e9,
        "stages_ms": {n: T.mean_ms(n) for n in T.pairs},
    }


def time_rpb(pipe, steps, warmup):
    """The attention with the global relative position bias (hla_attn_fwd_rpb) on the
    workload's resident inputs taken as sequence-ordered, with the Hilbert order
    (identity for row-major patterns) and a seeded float32 table [heads, 2H-1, 2W-1];
    eager calls with an event pair around each."""
    hla, w = pipe.hla, pipe.w
    pat = w.pattern
    g = torch.Generator(device="cpu")
    g.manual_seed(w.seed + 2000)
    table = torch.randn((w.heads, 2 * pat.H - 1, 2 * pat.W - 1), generator=g).cuda()
    if pat.hilbert:
        order = hla.hilbert_perm(pat.H, pat.W)[0]
    else:
        order = torch.arange(w.N, dtype=torch.int32, device="cuda")
    mask = hla.BlockMask(pat, w.tile_m, w.tile_n, totals=False).build()
    T = Timer()

    def call(i):
        s = pipe.sets[i % pipe.nsets]
        with T.stage("attn_rpb"):
            hla.attn_fwd_rpb(s["q"], s["k"], s["v"], order, table, mask, w.scale,
                             out=s["o"], lse=s["lse"])
    for i in range(warmup):
        call(i)
    torch.cuda.synchronize()
    T.active = True
    for i in range(steps):
        call(warmup + i)
    torch.cuda.synchronize()
    ms = T.mean_ms("attn_rpb")
    flops = pipe.tile_flops()[0]
    peak = BF16_PEAK_TFLOPS if w.dtype == "bf16" else FP32_PEAK_TFLOPS
    return {"attn_rpb_ms_per_call": ms,
            "attn_rpb_tflops_nonempty_tiles": flops / (ms * 1e-3) / 1e12,
            "attn_rpb_pct_peak": 100.0 * flops / (ms * 1e-3) / 1e12 / peak}


def summarize(pipe, timing):
    ms_step, eager_ms, passes = timing
    T = pipe.timer
    flops, tf, tp = pipe.tile_flops()
    w = pipe.w
    attn_ms = T.mean_ms("attn")
    attn_tflops = flops / (attn_ms * 1e-3) / 1e12
    peak = BF16_PEAK_TFLOPS if getattr(w, "dtype", "bf16") == "bf16" else FP32_PEAK_TFLOPS
    res = {
        "workload": w.name,
        "ms_per_step": ms_step,
        "ms_per_step_eager": eager_ms,
        "ms_per_step_graph": passes["graph"],
        "ms_per_step_stream": passes["stream"],
        "step_timing": "graph" if passes["graph"] <= passes["stream"] else "stream",
        "attn_ms": attn_ms,
        "attn_tile_tflops": attn_tflops,
        "attn_pct_peak": 100.0 * attn_tflops / peak,
        "attn_hbm_gbs": pipe.attn_bytes() / (attn_ms * 1e-3) / 1e9,
        "tiles_full": tf, "tiles_partial": tp,
        "tile_flops": flops,
        "stages_ms": {n: T.mean_ms(n) for n in T.pairs},
    }
    if "gather" in T.pairs:
        per = 1 if isinstance(w, W.LayerWorkload) else 3
        res["gather_gbs"] = per * pipe.perm_bytes_per_tensor() / (T.mean_ms("gather") * 1e-3) / 1e9
    if "scatter" in T.pairs:
        res["scatter_gbs"] = pipe.perm_bytes_per_tensor() / (T.mean_ms("scatter") * 1e-3) / 1e9
    return res


# ----------------------------------------------------------------------------
# one record per measured configuration


STEP_TEXT = {
    "attn_fwd_hilbert": "Hilbert index, tile lists and attention with the reordering fused in, in one "
                        "launch (hla_attn_fwd_hilbert)",
    "attn_fwd_perm": "Hilbert index and tile lists (one launch), attention with the reordering fused in "
                     "(hla_attn_fwd_perm)",
    "attn_fwd": "tile lists, attention",
}


def attn_config_record(w, hla, steps, warmup, fused_step=True):
    """A configuration's numbers: its step (for Hilbert patterns the reordering fused
    into the attention, else the plain attention), the attention kernel alone
    (back-to-back launches) with its roofline, and the gather / scatter kernels of
    the composed step with theirs."""
    n = max(steps, 20)
    rec = {"description": w.description, "pattern": w.pattern.kind, "B": w.B, "heads": w.heads,
           "tokens": w.N, "head_dim": w.d, "dtype": w.dtype, "tile": [w.tile_m, w.tile_n]}
    comp = make_pipeline(w, hla)
    rc = summarize(comp, run_timed(comp, steps, warmup))
    kms_c = comp.kernel_ms(n)
    flops, tf, tp = comp.tile_flops()
    nbytes = comp.attn_bytes()
    rec["tiles"] = {"full": tf, "partial": tp}
    rec["tile_flops"] = flops
    if comp.hilbert:
        pb = comp.perm_bytes_per_tensor()
        rec["perm"] = {"gather": perm_record(comp.perm_kernel_ms(n), pb,
                                             profile_traffic(f"permute_rows_gather_{w.name}", PERM_SOURCES)),
                       "scatter": perm_record(comp.perm_kernel_ms(n, scatter=True), pb,
                                              profile_traffic(f"permute_rows_scatter_{w.name}", PERM_SOURCES))}
    rec["composed_step"] = {"ms_per_step": rc["ms_per_step"], "ms_per_step_eager": rc["ms_per_step_eager"],
                            "attn_kernel_ms": kms_c, "value": flops / (rc["ms_per_step"] * 1e-3) / 1e12}
    del comp
    torch.cuda.empty_cache()
    res, kms, kernel = rc, kms_c, "attn_fwd"
    if w.pattern.hilbert and fused_step:
        fp = make_pipeline(w, hla, fused=True)
        res = summarize(fp, run_timed(fp, steps, warmup))
        kms, kernel = fp.kernel_ms(n), "attn_fwd_perm"
        del fp
        torch.cuda.empty_cache()
        if single_ok(w):
            rec["fused_step"] = {"ms_per_step": res["ms_per_step"],
                                 "ms_per_step_eager": res["ms_per_step_eager"],
                                 "attn_kernel_ms": kms,
                                 "value": flops / (res["ms_per_step"] * 1e-3) / 1e12}
            sp = make_pipeline(w, hla, single=True)
            res = summarize(sp, run_timed(sp, steps, warmup))
            kms, kernel = sp.kernel_ms(n), "attn_fwd_hilbert"
            del sp
            torch.cuda.empty_cache()
    peak = BF16_PEAK_TFLOPS if w.dtype == "bf16" else FP32_PEAK_TFLOPS
    rec.update({
        "step": STEP_TEXT[kernel],
        "ms_per_step": res["ms_per_step"], "ms_per_step_eager": res["ms_per_step_eager"],
        "value": flops / (res["ms_per_step"] * 1e-3) / 1e12, "unit": "TFLOP/s",
        "attn_ms_per_call": kms,
        "attn_tflops_nonempty_tiles": flops / (kms * 1e-3) / 1e12,
        "attn_pct_peak": 100.0 * flops / (kms * 1e-3) / 1e12 / peak,
        "peak_tflops": peak,
        "roofline": roofline_record(kernel, kms, nbytes, flops, w.dtype),
        "stages_ms": res["stages_ms"],
    })
    return rec


def layer_config_record(w, hla, steps, warmup):
    """The layer: its step (reordering fused into the projections), each kernel alone
    with its roofline, and the feature gather / scatter of the unfused step."""
    n = max(steps, 20)
    rec = {"description": w.description, "B": w.B, "heads": w.heads, "tokens": w.N,
           "head_dim": w.d, "embed": w.C, "dtype": "bf16", "tile": [w.tile_m, w.tile_n],
           "half_width": w.half_width}
    un = LayerPipeline(w, hla, fused=False)
    ru = summarize(un, run_timed(un, steps, warmup))
    pb = un.perm_bytes_per_tensor()
    rec["perm"] = {"gather": perm_record(un.kernel_ms("gather", n), pb),
                   "scatter": perm_record(un.kernel_ms("scatter", n), pb)}
    rec["unfused_step"] = {"ms_per_step": ru["ms_per_step"], "ms_per_step_eager": ru["ms_per_step_eager"]}
    del un
    torch.cuda.empty_cache()
    fused_res = None
    if single_ok(w):
        fp = LayerPipeline(w, hla, fused=True)
        fr = summarize(fp, run_timed(fp, steps, warmup))
        fused_res = {"ms_per_step": fr["ms_per_step"], "ms_per_step_eager": fr["ms_per_step_eager"],
                     "attn_kernel_ms": fp.kernel_ms("attn", n)}
        del fp
        torch.cuda.empty_cache()
    lp = LayerPipeline(w, hla, fused=True, single=single_ok(w))
    res = summarize(lp, run_timed(lp, steps, warmup))
    flops, tf, tp = lp.tile_flops()
    kernels = {}
    names = (("qkv", "qkv_proj"), ("attn", "attn_fwd_hilbert"), ("proj", "out_proj")) if lp.single else \
        (("qkv", "qkv_proj_perm"), ("attn", "attn_fwd"), ("proj", "out_proj_perm"))
    for which, name in names:
        ms = lp.kernel_ms(which, n)
        if which == "attn":
            nb, fl = lp.attn_bytes(), flops
        else:
            nb, fl = lp.proj_figures(which)
        kernels[which] = roofline_record(name, ms, nb, fl, "bf16")
        proj_name = f"proj_stream_{'qkv' if which == 'qkv' else 'out'}{'_plain' if lp.single else ''}_{w.name}"
        kernels[which]["traffic"] = (measured_traffic(w.name, name) if which == "attn" else
                                     profile_traffic(proj_name, PROJ_SOURCES))
    att = kernels["attn"]["kernel_ms_per_launch"]
    rec.update({
        "step": ("QKV projection, attention with the Hilbert rows and tile lists computed in the kernel "
                 "(hla_attn_fwd_hilbert), output projection: three launches, all in grid order"
                 if lp.single else
                 "Hilbert index and tile lists (one launch), QKV projection with the gather fused in, "
                 "attention, output projection with the scatter fused in"),
        "ms_per_step": res["ms_per_step"], "ms_per_step_eager": res["ms_per_step_eager"],
        "value": flops / (res["ms_per_step"] * 1e-3) / 1e12, "unit": "TFLOP/s",
        "tiles": {"full": tf, "partial": tp}, "tile_flops": flops,
        "attn_ms_per_call": att,
        "attn_tflops_nonempty_tiles": flops / (att * 1e-3) / 1e12,
        "attn_pct_peak": 100.0 * flops / (att * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
        "roofline": max(kernels.values(), key=lambda r: r["kernel_ms_per_launch"]),
        "kernels": kernels, "stages_ms": res["stages_ms"],
    })
    if fused_res is not None:
        rec["fused_step"] = fused_res
    del lp
    torch.cuda.empty_cache()
    return rec


def hilbert_index_record(hla, side, n):
    """hla_hilbert_perm on a side x side grid: order and rank (8 bytes per cell
    written), n back-to-back launches."""
    N = side * side
    order = torch.empty(N, dtype=torch.int32, device="cuda")
    rank = torch.empty(N, dtype=torch.int32, device="cuda")
    ms = b2b_ms(lambda i: hla.hilbert_perm(side, side, out=(order, rank)), n)
    gbs = 8 * N / (ms * 1e-3) / 1e9
    return {"grid": [side, side], "tokens": N, "ms_per_call": ms, "bytes_written": 8 * N,
            "gbs": gbs, "frac": gbs / HBM_PEAK_GBS}


# ----------------------------------------------------------------------------
# CPU baseline: the oracle on a bounded sample of the same step


def blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        n = [i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"]
        return max(n) if n else 1
    except Exception:
        return 1


def cpu_baseline(w: W.AttnWorkload, flops_per_step: float, budget_s: float = 12.0):
    """Times the oracle's stages for one step of workload w: Hilbert order, gather of
    q, k, v, brute-force tile lists, dense masked attention on a sample of query rows
    (scaled to all rows), scatter. Returns the record for the JSON line."""
    import numpy as np

    from oracle import attention as o_attn
    from oracle import blockmask as o_bm
    from oracle import hilbert as o_hil
    from oracle import permute as o_perm

    q, k, v = (t.float().numpy().astype(np.float64) for t in W.workload_inputs(w))
    pat = w.pattern
    t0 = time.perf_counter()
    order = o_hil.hilbert_order(pat.H, pat.W)
    t_hil = time.perf_counter() - t0
    t0 = time.perf_counter()
    qh, kh, vh = (o_perm.gather(a, order) for a in (q, k, v))
    t_gather = time.perf_counter() - t0
    # tile lists: brute force over a sample of query-tile rows, scaled to all rows
    nq = w.N // w.tile_m
    rows_t = list(range(0, nq, max(1, nq // 16)))
    t0 = time.perf_counter()
    o_bm.build(pat, w.tile_m, w.tile_n, rows_t)
    t_mask = (time.perf_counter() - t0) * nq / len(rows_t)
    # attention: calibrate the row sample on a pilot, then time the sample
    # (the second pilot: the first one's time includes first-touch costs that the
    # sample does not pay again)
    pilot = np.arange(0, w.N, max(1, w.N // 16))[:16]
    for _ in range(2):
        t0 = time.perf_counter()
        o_attn.attention(qh, kh, vh, pat, w.scale, rows=pilot)
        per_row = (time.perf_counter() - t0) / len(pilot)
    n_rows = int(max(16, min(w.N, budget_s / max(per_row, 1e-9))))
    rows = np.linspace(0, w.N - 1, n_rows).astype(np.int64)
    t0 = time.perf_counter()
    out, _ = o_attn.attention(qh, kh, vh, pat, w.scale, rows=rows)
    t_attn = (time.perf_counter() - t0) * w.N / n_rows
    t0 = time.perf_counter()
    o_perm.scatter(qh, order)   # same-size scatter
    t_scatter = time.perf_counter() - t0
    total = t_hil + t_gather + t_mask + t_attn + t_scatter
    return {
        "value": flops_per_step / total / 1e12,
        "unit": "TFLOP/s",
        "cores": blas_threads(),
        "kind": "oracle",
        "sample": (f"float64 oracle on the host: full Hilbert order and gathers, brute-force tile "
                   f"lists on {len(rows_t)}/{nq} query-tile rows, dense masked attention on "
                   f"{n_rows}/{w.N} query rows of all {w.B * w.heads} (b,h); each sampled stage "
                   f"scaled to the whole step; est. {total:.1f} s per step"),
        "stage_s": {"hilbert": t_hil, "gather": t_gather, "mask": t_mask, "attn": t_attn,
                    "scatter": t_scatter},
        "host": {"cpu_count": os.cpu_count(),
                 "affinity": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None,
                 "processor": platform.processor() or platform.machine()},
    }


# ----------------------------------------------------------------------------


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=W.C3.name, choices=sorted(W.WORKLOADS))
    ap.add_argument("--compare", default=None,
                    help="workload timed through the same kernel for the row-major comparison")
    ap.add_argument("--all", action="store_true",
                    help="also time every workload (each one's results on stderr)")
    ap.add_argument("--all-out", default=None,
                    help="with --all, also write every workload's results to this JSON file")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-backward", action="store_true",
                    help="skip timing the backward pass of the workload")
    ap.add_argument("--no-rpb", action="store_true",
                    help="skip timing the attention with the relative position bias")
    ap.add_argument("--step", default="single", choices=["single", "fused", "composed", "composed-only"],
                    help="which step of a Hilbert workload the headline value times: the whole "
                         "step in one launch (hla_attn_fwd_hilbert; on 2^k x 2^k grids, else as "
                         "fused), the reordering fused into the attention after one index-and-lists "
                         "launch (hla_attn_fwd_perm), or separate gather / attention / scatter "
                         "calls; the others are reported beside it (composed-only: skip the fused "
                         "steps)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-configuration records (every measured workload's step, "
                         "attention kernel, gather / scatter kernels and rooflines) and the "
                         "Hilbert index at 4096 x 4096")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="before the steps, time a plain device-to-device copy of this many MiB "
                         "(a kernel of known traffic, to calibrate HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the hot path is "
              f"measured on one GPU's share and has no multi-GPU launch.", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)

    import paper_2511_05832_amd as hla
    hla.lib()
    torch.cuda.set_device(0)

    if args.copy_mib:
        src = torch.empty(args.copy_mib << 20, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] copied {args.copy_mib} MiB x 5", file=sys.stderr, flush=True)
        del src, dst

    w = W.WORKLOADS[args.workload]
    pipe = make_pipeline(w, hla)
    timing = run_timed(pipe, args.steps, args.warmup)
    res = summarize(pipe, timing)
    if isinstance(w, W.AttnWorkload):
        res["attn_kernel_ms"] = pipe.kernel_ms(max(args.steps, 20))
    else:
        res["attn_kernel_ms"] = pipe.kernel_ms("attn", max(args.steps, 20))
    print(f"[bench] {w.name} (composed): {json.dumps(res)}", file=sys.stderr, flush=True)
    bwd = None
    if isinstance(w, W.AttnWorkload) and not args.no_backward:
        bwd = time_backward(pipe, args.steps, args.warmup)
        print(f"[bench] {w.name} backward: {json.dumps(bwd)}", file=sys.stderr, flush=True)
    # The same step with the reordering fused into the attention (Hilbert patterns).
    res_fused = bwd_fused = None
    if isinstance(w, W.AttnWorkload) and w.pattern.hilbert and args.step != "composed-only":
        del pipe
        torch.cuda.empty_cache()
        fpipe = make_pipeline(w, hla, fused=True)
        res_fused = summarize(fpipe, run_timed(fpipe, args.steps, args.warmup))
        res_fused["attn_kernel_ms"] = fpipe.kernel_ms(max(args.steps, 20))
        print(f"[bench] {w.name} (fused): {json.dumps(res_fused)}", file=sys.stderr, flush=True)
        if not args.no_backward:
            bwd_fused = time_backward(fpipe, args.steps, args.warmup)
            print(f"[bench] {w.name} backward (fused): {json.dumps(bwd_fused)}", file=sys.stderr, flush=True)
        pipe = fpipe   # the algorithmic figures below depend on the workload only
    # The whole step as one launch (index, lists and reordered attention inside
    # hla_attn_fwd_hilbert), where the workload allows it.
    res_single = None
    if (isinstance(w, W.AttnWorkload) and single_ok(w) and args.step in ("single", "fused")
            and res_fused is not None):
        spipe = make_pipeline(w, hla, single=True)
        res_single = summarize(spipe, run_timed(spipe, args.steps, args.warmup))
        res_single["attn_kernel_ms"] = spipe.kernel_ms(max(args.steps, 20))
        print(f"[bench] {w.name} (single launch): {json.dumps(res_single)}", file=sys.stderr, flush=True)
        del spipe
        torch.cuda.empty_cache()
    rpb = None
    if isinstance(w, W.AttnWorkload) and not args.no_rpb:
        rpb = time_rpb(pipe, args.steps, args.warmup)
        print(f"[bench] {w.name} with the position bias: {json.dumps(rpb)}", file=sys.stderr, flush=True)
    res_composed = res
    if args.step == "single" and res_single:
        res = res_single
    elif args.step in ("single", "fused") and res_fused:
        res = res_fused
    ms = res["ms_per_step"]
    attn_kernel = ("attn_fwd_hilbert" if res is res_single or getattr(pipe, "single", False) and
                   isinstance(w, W.LayerWorkload) else
                   "attn_fwd_perm" if res is res_fused else "attn_fwd")

    compare = args.compare
    if compare is None and not args.copy_mib:
        compare = {W.C3.name: W.C3_ROWMAJOR.name, W.C4.name: W.C4_ROWMAJOR.name}.get(w.name)
    cmp_res = None
    if compare:
        cpipe = make_pipeline(W.WORKLOADS[compare], hla)
        cmp_res = summarize(cpipe, run_timed(cpipe, args.steps, args.warmup))
        print(f"[bench] {compare}: {json.dumps(cmp_res)}", file=sys.stderr, flush=True)
        del cpipe

    if args.all:
        allres = {}
        for name, wl in W.WORKLOADS.items():
            p = make_pipeline(wl, hla)
            r = summarize(p, run_timed(p, args.steps, args.warmup))
            if isinstance(wl, W.AttnWorkload) and not args.no_backward:
                r["backward"] = time_backward(p, args.steps, args.warmup)
            allres[name] = r
            print(f"[bench] {name}: {json.dumps(r)}", file=sys.stderr, flush=True)
            del p
            torch.cuda.empty_cache()
        if args.all_out:
            os.makedirs(os.path.dirname(os.path.abspath(args.all_out)), exist_ok=True)
            with open(args.all_out, "w") as f:
                json.dump(allres, f, indent=1)

    configs, hilbert_index = None, None
    if not args.no_configs and not args.copy_mib:
        configs = {}
        for cw in (W.C1, W.C2, W.C3, W.C3_ROWMAJOR, W.C4, W.C4_ROWMAJOR, W.C5):
            if isinstance(cw, W.LayerWorkload):
                configs[cw.name] = layer_config_record(cw, hla, args.steps, args.warmup)
            else:
                configs[cw.name] = attn_config_record(cw, hla, args.steps, args.warmup)
            print(f"[bench] config {cw.name}: {json.dumps(configs[cw.name])}", file=sys.stderr, flush=True)
        # the index at the configurations' sizes is launch-bound; at 4096 x 4096
        # (16.8 M cells, 128 MiB written) its GB/s means something
        hilbert_index = {f"{sd}x{sd}": hilbert_index_record(hla, sd, max(args.steps, 20))
                         for sd in (128, 256, 4096)}
        print(f"[bench] hilbert index: {json.dumps(hilbert_index)}", file=sys.stderr, flush=True)

    flops = res["tile_flops"]
    # the dominant kernel's average duration: back-to-back launches between one
    # event pair where measured, else the eager pass's per-stage events
    attn_s = res.get("attn_kernel_ms", res["attn_ms"]) * 1e-3
    is_bf16 = getattr(w, "dtype", "bf16") == "bf16"
    # dominant kernel: attention. HBM-bound when its bytes take longer at peak than
    # its tile FLOPs do on the matrix cores.
    t_hbm = pipe.attn_bytes() / (HBM_PEAK_GBS * 1e9)
    t_mfma = flops / ((BF16_PEAK_TFLOPS if is_bf16 else FP32_PEAK_TFLOPS) * 1e12)
    peak_tf = BF16_PEAK_TFLOPS if is_bf16 else FP32_PEAK_TFLOPS
    kernel_tflops = flops / attn_s / 1e12
    if t_hbm >= t_mfma:
        achieved = pipe.attn_bytes() / attn_s / 1e9
        roofline = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic(w.name, attn_kernel),
                    "kernel": attn_kernel, "kernel_ms_per_launch": attn_s * 1e3,
                    "algorithmic_bytes": pipe.attn_bytes(),
                    "mfma_frac": kernel_tflops / peak_tf}
    else:
        roofline = {"bound": "mfma", "achieved": kernel_tflops, "peak": peak_tf,
                    "unit": "TFLOP/s", "frac": kernel_tflops / peak_tf,
                    "traffic": measured_traffic(w.name, attn_kernel),
                    "kernel": attn_kernel, "kernel_ms_per_launch": attn_s * 1e3,
                    "algorithmic_flops": flops,
                    "hbm_frac": pipe.attn_bytes() / attn_s / 1e9 / HBM_PEAK_GBS}

    cpu = None
    if not args.no_cpu_baseline and isinstance(w, W.AttnWorkload):
        cpu = cpu_baseline(w, flops)

    line = {
        "metric": METRIC,
        "value": flops / (ms * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "ms_per_step_eager": res["ms_per_step_eager"],
        "timing": "ms_per_step: the faster of two timings of the same K steps, replayed from "
                  "HIP graphs (one per input set; ms_per_step_graph) or launched back to back "
                  "from the host with no event between steps (ms_per_step_stream); "
                  "step_timing names it. Per-kernel times from an eager pass of the same "
                  "steps with events around every stage (ms_per_step_eager: its median "
                  "step); the roofline's kernel time from back-to-back launches of that "
                  "kernel alone between one event pair",
        "ms_per_step_graph": res["ms_per_step_graph"],
        "ms_per_step_stream": res["ms_per_step_stream"],
        "step_timing": res["step_timing"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": getattr(w, "dtype", "bf16"),
        "data": "synthetic",
        "config": {"workload": w.name, "description": w.description,
                   "B": w.B, "heads": w.heads, "tokens": w.N, "head_dim": w.d,
                   "tile": [w.tile_m, w.tile_n], "parallelism": "single-gpu"},
        "step": (("QKV projection, attention with the Hilbert rows and tile lists computed in the "
                  "kernel (hla_attn_fwd_hilbert), output projection: three launches, all in grid order"
                  if getattr(pipe, "single", False) else
                  "Hilbert index and tile lists (one launch), QKV projection with the gather fused "
                  "in, attention, output projection with the scatter fused in")
                 if isinstance(w, W.LayerWorkload) else
                 STEP_TEXT[attn_kernel] if attn_kernel != "attn_fwd" else
                 "Hilbert index and tile lists (one launch), gather of q/k/v, attention, scatter of out"
                 if getattr(getattr(w, "pattern", None), "hilbert", False) else
                 "tile lists, attention"),
        "attn_ms_per_call": res["attn_ms"],
        "attn_tflops_nonempty_tiles": res["attn_tile_tflops"],
        "attn_pct_bf16_peak": res["attn_pct_peak"],
        "perm_gbs": {"gather": res_composed.get("gather_gbs"),
                     "scatter": res_composed.get("scatter_gbs"),
                     "note": "eager step's stage events (three gathers, one scatter)"},
        "stages_ms": res["stages_ms"],
        "tiles": {"full": res["tiles_full"], "partial": res["tiles_partial"]},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    for key, other in (("single_step", res_single), ("fused_step", res_fused),
                       ("composed_step", res_composed)):
        if other and other is not res:
            line[key] = {
                "ms_per_step": other["ms_per_step"], "ms_per_step_eager": other["ms_per_step_eager"],
                "value": flops / (other["ms_per_step"] * 1e-3) / 1e12,
                "attn_ms_per_call": other["attn_ms"], "stages_ms": other["stages_ms"]}
            if "attn_kernel_ms" in other:
                line[key]["attn_kernel_ms"] = other["attn_kernel_ms"]
    if configs and w.name in configs and "perm" in configs[w.name]:
        pr = configs[w.name]["perm"]
        line["perm_gbs"].update({
            "gather_kernel": pr["gather"]["gbs"], "gather_frac": pr["gather"]["frac"],
            "scatter_kernel": pr["scatter"]["gbs"], "scatter_frac": pr["scatter"]["frac"],
            "kernel_note": "one [B, heads, N, d] tensor per launch, back-to-back launches; "
                           "frac = achieved / 8 TB/s"})
    if configs:
        line["configs"] = configs
    if hilbert_index:
        line["hilbert_index"] = hilbert_index
    if bwd:
        line["backward"] = bwd
    if bwd_fused:
        line["backward_fused"] = bwd_fused
    if rpb:
        line["rpb"] = rpb
    if cmp_res:
        line["rowmajor_comparison"] = {
            "workload": cmp_res["workload"], "attn_ms_per_call": cmp_res["attn_ms"],
            "tiles": {"full": cmp_res["tiles_full"], "partial": cmp_res["tiles_partial"]},
            "hilbert_speedup_attn": cmp_res["attn_ms"] / res["attn_ms"]}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
