// Tile classification and per-row / per-column tile lists (Sec. 3.1: full, partial and
// empty blocks of the N x N score matrix; empty blocks are skipped, full
// blocks run without a mask, partial blocks need the element mask).
//
// Exact closed-form classification, one thread per (query tile, key tile):
// a tile covers an interval of query positions and an interval of key
// positions. For the 1-D patterns the allowed pairs of an interval pair are
// decided per axis from interval end points (window ids, band distances,
// clamped neighbourhood starts). For the 2-D row-major patterns a position
// interval is split into at most three grid rectangles (a partial first row,
// whole middle rows, a partial last row); the pattern is a product of a row
// condition and a column condition, so each rectangle pair is decided per axis
// and the tile is non-empty if any pair is, full if every pair is.
//
// Ragged tilings (N not a multiple of a tile): the last tile row / column covers
// the positions up to N - 1 and padded slots past them, which are never allowed;
// such a tile is classified on its real positions and is never full.
//
// Layout: one workgroup per line walks the tiles of that line in chunks of 256,
// compacts full and partial indices with wave ballots into ascending lists,
// then pads the rest of both lists with -1. A line is a query-tile row (the
// forward pass and the query gradients walk these) or, for the optional
// transposed lists, a key-tile column (the key and value gradients walk these).
#include "hilbert_common.h"

namespace hla {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

struct Cls {
  bool any, all;
};

enum AxisKind { AX_WINDOW, AX_SLIDE, AX_NEIGH };

// Query interval [x0, x1] against key interval [y0, y1] on one axis.
//   AX_WINDOW: groups floor((x + off) / g); allowed iff same group
//   AX_SLIDE:  |x - y| <= g
//   AX_NEIGH:  y in [s(x), s(x) + g), s(x) = clamp(x - g/2, 0, extent - g)
__device__ __forceinline__ Cls axis_cls(int kind, int g, int off, int extent, int x0,
                                        int x1, int y0, int y1) {
  Cls c;
  if (kind == AX_WINDOW) {
    const int ga = (x0 + off) / g, gb = (x1 + off) / g;
    const int ha = (y0 + off) / g, hb = (y1 + off) / g;
    c.any = max(ga, ha) <= min(gb, hb);
    c.all = (ga == gb) && (ha == hb) && (ga == ha);
  } else if (kind == AX_SLIDE) {
    const int dmin = max(0, max(y0 - x1, x0 - y1));
    const int dmax = max(abs(x0 - y1), abs(x1 - y0));
    c.any = dmin <= g;
    c.all = dmax <= g;
  } else {
    const int s0 = min(max(x0 - g / 2, 0), extent - g);
    const int s1 = min(max(x1 - g / 2, 0), extent - g);
    c.any = (s0 <= y1) && (y0 <= s1 + g - 1);
    c.all = (s1 <= y0) && (y1 <= s0 + g - 1);
  }
  return c;
}

// A position interval [a, b] as up to three grid rectangles in fixed slots:
// 0 = the first row's part, 1 = the whole rows between (if any), 2 = the last
// row's part (if it is not the first row). Fixed slots keep every field in
// registers (an array filled at a running index would live in scratch memory).
struct Rects {
  bool ok[3];
  int r0[3], r1[3], c0[3], c1[3];
};

__device__ __forceinline__ Rects split_rows(int a, int b, int W) {
  Rects R;
  const int ra = a / W, ca = a - ra * W;
  const int rb = b / W, cb = b - rb * W;
  const bool one_row = ra == rb;
  R.ok[0] = true;
  R.r0[0] = ra; R.r1[0] = ra; R.c0[0] = ca; R.c1[0] = one_row ? cb : W - 1;
  R.ok[1] = rb - ra >= 2;
  R.r0[1] = ra + 1; R.r1[1] = rb - 1; R.c0[1] = 0; R.c1[1] = W - 1;
  R.ok[2] = !one_row;
  R.r0[2] = rb; R.r1[2] = rb; R.c0[2] = 0; R.c1[2] = cb;
  return R;
}

__device__ int classify_tile(const PatternArgs &p, int i0, int i1, int j0, int j1) {
  switch (p.kind) {
    case HLA_HILBERT_WINDOW: {
      Cls c = axis_cls(AX_WINDOW, p.p0, 0, p.N, i0, i1, j0, j1);
      return c.all ? 2 : (c.any ? 1 : 0);
    }
    case HLA_HILBERT_SHIFTED_WINDOW: {
      Cls c = axis_cls(AX_WINDOW, p.p0, p.p0 - p.p1, p.N, i0, i1, j0, j1);
      return c.all ? 2 : (c.any ? 1 : 0);
    }
    case HLA_HILBERT_SLIDE: {
      Cls c = axis_cls(AX_SLIDE, p.p0, 0, p.N, i0, i1, j0, j1);
      return c.all ? 2 : (c.any ? 1 : 0);
    }
    case HLA_HILBERT_NEIGHBORHOOD: {
      Cls c = axis_cls(AX_NEIGH, p.p0, 0, p.N, i0, i1, j0, j1);
      return c.all ? 2 : (c.any ? 1 : 0);
    }
    default:
      break;
  }
  const int ax = p.kind == HLA_ROWMAJOR_WINDOW ? AX_WINDOW
                 : p.kind == HLA_ROWMAJOR_SLIDE ? AX_SLIDE
                                                : AX_NEIGH;
  const Rects Q = split_rows(i0, i1, p.W);
  const Rects K = split_rows(j0, j1, p.W);
  bool any = false, all = true;
#pragma unroll
  for (int a = 0; a < 3; ++a) {
#pragma unroll
    for (int b = 0; b < 3; ++b) {
      if (!Q.ok[a] || !K.ok[b]) continue;
      const Cls cr = axis_cls(ax, p.p0, 0, p.H, Q.r0[a], Q.r1[a], K.r0[b], K.r1[b]);
      const Cls cc = axis_cls(ax, p.p1, 0, p.W, Q.c0[a], Q.c1[a], K.c0[b], K.c1[b]);
      any = any || (cr.any && cc.any);
      all = all && (cr.all && cc.all);
    }
  }
  return all ? 2 : (any ? 1 : 0);
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// COLS = false: line = query-tile row q, entries = key tiles.
// COLS = true:  line = key-tile column k, entries = query tiles.
// PATH: the grid carries `path.blocks` more workgroups after the lines, which
// compute the Hilbert index of the same launch (hla_build_path_and_mask): the two
// jobs are independent, and one launch is one graph node instead of two.
template <bool COLS, bool PATH>
__global__ void __launch_bounds__(kThreads)
    classify_lines(PatternArgs p, int32_t tile_m, int32_t tile_n, int32_t n_entries,
                   int32_t *__restrict__ n_full, int32_t *__restrict__ full_idx,
                   int32_t *__restrict__ n_part, int32_t *__restrict__ part_idx,
                   HilbertJob path) {
  if constexpr (PATH) {
    const int32_t b = (int32_t)blockIdx.x - ((int32_t)gridDim.x - path.blocks);
    if (b >= 0) {   // uniform over the workgroup: it leaves before any barrier
      hilbert4_block(path, b, (int32_t)threadIdx.x);
      return;
    }
  }
  __shared__ int32_t wave_f[kWaves], wave_p[kWaves];
  const int line = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int32_t *flist = full_idx + (int64_t)line * n_entries;
  int32_t *plist = part_idx + (int64_t)line * n_entries;
  int nf = 0, np = 0;
  for (int base = 0; base < n_entries; base += kThreads) {
    const int e = base + tid;
    int cls = 0;
    if (e < n_entries) {
      const int qt = COLS ? e : line, kt = COLS ? line : e;
      // Ragged edge: the tile's real positions end at N - 1; the padded slots are
      // never allowed, so a tile reaching past N is never full.
      const int i1 = qt * tile_m + tile_m - 1, j1 = kt * tile_n + tile_n - 1;
      cls = classify_tile(p, qt * tile_m, min(i1, p.N - 1), kt * tile_n, min(j1, p.N - 1));
      if (cls == 2 && (i1 >= p.N || j1 >= p.N)) cls = 1;
    }
    const uint64_t bf = __ballot(cls == 2);
    const uint64_t bp = __ballot(cls == 1);
    if (lane == 0) {
      wave_f[wave] = __popcll(bf);
      wave_p[wave] = __popcll(bp);
    }
    __syncthreads();
    int off_f = 0, off_p = 0, tot_f = 0, tot_p = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      if (w < wave) {
        off_f += wave_f[w];
        off_p += wave_p[w];
      }
      tot_f += wave_f[w];
      tot_p += wave_p[w];
    }
    if (cls == 2) flist[nf + off_f + lanes_below(bf)] = e;
    if (cls == 1) plist[np + off_p + lanes_below(bp)] = e;
    nf += tot_f;
    np += tot_p;
    __syncthreads();
  }
  for (int t = nf + tid; t < n_entries; t += kThreads) flist[t] = -1;
  for (int t = np + tid; t < n_entries; t += kThreads) plist[t] = -1;
  if (tid == 0) {
    n_full[line] = nf;
    n_part[line] = np;
  }
}

__global__ void __launch_bounds__(kThreads)
    sum_totals(const int32_t *__restrict__ n_full, const int32_t *__restrict__ n_part,
               int32_t n, int32_t *__restrict__ totals) {
  __shared__ int32_t sf[kWaves], sp[kWaves];
  int f = 0, p = 0;
  for (int i = threadIdx.x; i < n; i += kThreads) {
    f += n_full[i];
    p += n_part[i];
  }
  for (int o = 32; o > 0; o >>= 1) {
    f += __shfl_xor(f, o);
    p += __shfl_xor(p, o);
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sf[wave] = f;
    sp[wave] = p;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int tf = 0, tp = 0;
    for (int w = 0; w < kWaves; ++w) {
      tf += sf[w];
      tp += sp[w];
    }
    totals[0] = tf;
    totals[1] = tp;
  }
}

}  // namespace

hipError_t launch_block_mask(const PatternArgs &pat, int32_t tile_m, int32_t tile_n,
                             int32_t n_qtiles, int32_t n_ktiles, const BlockLists &rows,
                             const BlockLists *cols, int32_t *totals, hipStream_t s,
                             const HilbertJob *path) {
  if (path && path->blocks > 0) {
    hipLaunchKernelGGL((classify_lines<false, true>), dim3(n_qtiles + path->blocks), dim3(kThreads),
                       0, s, pat, tile_m, tile_n, n_ktiles, rows.n_full, rows.full_idx, rows.n_part,
                       rows.part_idx, *path);
  } else {
    hipLaunchKernelGGL((classify_lines<false, false>), dim3(n_qtiles), dim3(kThreads), 0, s, pat,
                       tile_m, tile_n, n_ktiles, rows.n_full, rows.full_idx, rows.n_part,
                       rows.part_idx, HilbertJob{});
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (cols) {
    hipLaunchKernelGGL((classify_lines<true, false>), dim3(n_ktiles), dim3(kThreads), 0, s, pat,
                       tile_m, tile_n, n_qtiles, cols->n_full, cols->full_idx, cols->n_part,
                       cols->part_idx, HilbertJob{});
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (!totals) return hipSuccess;
  hipLaunchKernelGGL(sum_totals, dim3(1), dim3(kThreads), 0, s, rows.n_full, rows.n_part,
                     n_qtiles, totals);
  return hipGetLastError();
}

hipError_t launch_path_and_mask(int32_t side, int32_t *order, int32_t *rank,
                                const PatternArgs &pat, int32_t tile_m, int32_t tile_n,
                                int32_t n_qtiles, int32_t n_ktiles, const BlockLists &rows,
                                const BlockLists *cols, int32_t *totals, hipStream_t s) {
  int32_t lg = 0;
  while ((1 << lg) < side) ++lg;
  const HilbertJob job = make_hilbert_job(lg, order, rank);
  return launch_block_mask(pat, tile_m, tile_n, n_qtiles, n_ktiles, rows, cols, totals, s, &job);
}

}  // namespace hla
