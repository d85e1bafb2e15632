// Exact closed-form classification of one (query tile, key tile) pair of the
// N x N score matrix as empty (0), partial (1) or full (2) (Sec. 3.1: full,
// partial and empty blocks), shared by the tile-list builder and the attention
// that classifies its own row's tiles.
//
// A tile covers an interval of query positions and an interval of key
// positions. For the 1-D patterns the allowed pairs of an interval pair are
// decided per axis from interval end points (window ids, band distances,
// clamped neighbourhood starts). For the 2-D row-major patterns a position
// interval is split into at most three grid rectangles (a partial first row,
// whole middle rows, a partial last row); the pattern is a product of a row
// condition and a column condition, so each rectangle pair is decided per axis
// and the tile is non-empty if any pair is, full if every pair is.
#pragma once

#include "hla_internal.h"

namespace hla {

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

__device__ __forceinline__ int classify_tile(const PatternArgs &p, int i0, int i1, int j0, int j1) {
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

// The same for the 1-D (Hilbert) patterns only: no row-major branch, for callers
// that only see those.
__device__ __forceinline__ int classify_tile_1d(const PatternArgs &p, int i0, int i1, int j0, int j1) {
  const int kind = p.kind == HLA_HILBERT_SLIDE ? AX_SLIDE
                   : p.kind == HLA_HILBERT_NEIGHBORHOOD ? AX_NEIGH
                                                        : AX_WINDOW;
  const int off = p.kind == HLA_HILBERT_SHIFTED_WINDOW ? p.p0 - p.p1 : 0;
  const Cls c = axis_cls(kind, p.p0, off, p.N, i0, i1, j0, j1);
  return c.all ? 2 : (c.any ? 1 : 0);
}

// Tile (qt, kt) of a tile_m x tile_n tiling. Ragged edge: the tile's real
// positions end at N - 1; the padded slots are never allowed, so a tile reaching
// past N is classified on its real positions and is never full.
template <bool ONE_D = false>
__device__ __forceinline__ int tile_class(const PatternArgs &p, int tile_m, int tile_n, int qt, int kt) {
  const int i1 = qt * tile_m + tile_m - 1, j1 = kt * tile_n + tile_n - 1;
  const int ci1 = min(i1, p.N - 1), cj1 = min(j1, p.N - 1);
  const int cls = ONE_D ? classify_tile_1d(p, qt * tile_m, ci1, kt * tile_n, cj1)
                        : classify_tile(p, qt * tile_m, ci1, kt * tile_n, cj1);
  return cls == 2 && (i1 >= p.N || j1 >= p.N) ? 1 : cls;
}

}  // namespace hla
