// Hilbert index device code shared by the index kernel (hilbert.hip) and the
// launch that builds the index and the tile lists together (blockmask.hip).
// Levels are walked from the coarsest down with the orientation of the current
// sub-square as two bits, sw (axes swapped) and fl (both axes reflected); see
// hilbert.hip for the curve's convention.
#pragma once

#include "hla_internal.h"

namespace hla {

// Orientation change on entering quadrant q (0..3 in visiting order): transpose
// for q = 0, anti-transpose for q = 3, none otherwise.
constexpr uint32_t turn_sw(uint32_t q) { return 1u ^ ((q ^ (q >> 1)) & 1u); }
constexpr uint32_t turn_fl(uint32_t q) { return q & (q >> 1) & 1u; }

// Levels lg-1 .. lo of curve position d: ORs the cell's x, y bits of those
// levels into x, y and leaves the orientation of the level-lo sub-square.
__device__ __forceinline__ void d2xy_levels(uint32_t d, int lg, int lo, uint32_t &x, uint32_t &y,
                                            uint32_t &sw, uint32_t &fl) {
  for (int l = lg - 1; l >= lo; --l) {
    const uint32_t q = (d >> (2 * l)) & 3u;
    uint32_t a = q >> 1, b = (q ^ a) & 1u;   // quadrant in the sub-curve's own frame
    const uint32_t t = ((a ^ b) & sw) ^ fl;  // into the grid's frame
    x |= (a ^ t) << l;
    y |= (b ^ t) << l;
    sw ^= turn_sw(q);
    fl ^= turn_fl(q);
  }
}

// Levels lg-1 .. lo of cell (x, y): ORs the curve digits of those levels into d.
__device__ __forceinline__ void xy2d_levels(uint32_t x, uint32_t y, int lg, int lo, uint32_t &d,
                                            uint32_t &sw, uint32_t &fl) {
  for (int l = lg - 1; l >= lo; --l) {
    uint32_t a = ((x >> l) & 1u) ^ fl, b = ((y >> l) & 1u) ^ fl;
    const uint32_t t = (a ^ b) & sw;
    a ^= t;
    b ^= t;
    const uint32_t q = (a << 1) | (a ^ b);
    d |= q << (2 * l);
    sw ^= turn_sw(q);
    fl ^= turn_fl(q);
  }
}

__device__ __forceinline__ void store4(int32_t *p, int32_t i4, const uint32_t (&v)[4], bool vec) {
  if (vec) {
    *reinterpret_cast<int4 *>(p + 4 * i4) = make_int4((int)v[0], (int)v[1], (int)v[2], (int)v[3]);
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) p[4 * i4 + j] = (int32_t)v[j];
  }
}

// The index on a side = 2^lg >= 4 square as 256-thread blocks: blocks
// [0, blocks_order) write order, the rest rank (either part may be absent);
// thread m of a part writes entries 4m .. 4m+3. vec: both outputs are 16-byte
// aligned.
struct HilbertJob {
  int32_t lg, n4, blocks_order, blocks;
  int32_t *order, *rank;
  int32_t vec;
};

inline HilbertJob make_hilbert_job(int32_t lg, int32_t *order, int32_t *rank) {
  HilbertJob j;
  j.lg = lg;
  j.n4 = (1 << (2 * lg)) / 4;
  const int32_t blocks = (j.n4 + 255) / 256;
  j.blocks_order = order ? blocks : 0;
  j.blocks = j.blocks_order + (rank ? blocks : 0);
  j.order = order;
  j.rank = rank;
  j.vec = ((reinterpret_cast<uintptr_t>(order) | reinterpret_cast<uintptr_t>(rank)) & 15u) == 0;
  return j;
}

// store4 with non-temporal 16-byte stores (the index kernel's outputs stream
// past the caches: 27.8 -> 25.5 us at 4096 x 4096).
typedef unsigned int u32x4h __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void store4nt(int32_t *p, int32_t i4, const uint32_t (&v)[4], bool vec) {
  if (vec) {
    const u32x4h w = {v[0], v[1], v[2], v[3]};
    __builtin_nontemporal_store(w, reinterpret_cast<u32x4h *>(p + 4 * i4));
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) p[4 * i4 + j] = (int32_t)v[j];
  }
}

// Block b (< job.blocks) of the job, thread tid (< 256).
__device__ __forceinline__ void hilbert4_block(const HilbertJob &job, int32_t b, int32_t tid) {
  const int32_t lg = job.lg, n4 = job.n4;
  const bool vec = job.vec != 0;
  uint32_t out[4];
  if (b < job.blocks_order) {
    const int32_t m = b * 256 + tid;
    if (m >= n4) return;
    uint32_t x = 0, y = 0, sw = 0, fl = 0;
    d2xy_levels(4u * (uint32_t)m, lg, 1, x, y, sw, fl);
#pragma unroll
    for (uint32_t j = 0; j < 4; ++j) {   // the last level: digit j
      const uint32_t a = j >> 1, b = (j ^ a) & 1u, t = ((a ^ b) & sw) ^ fl;
      out[j] = ((y | (b ^ t)) << lg) | (x | (a ^ t));
    }
    store4(job.order, m, out, vec);
  } else {
    const int32_t m = (b - job.blocks_order) * 256 + tid;
    if (m >= n4) return;
    const uint32_t t0 = 4u * (uint32_t)m;
    const uint32_t y = t0 >> lg, x0 = t0 & ((1u << lg) - 1u);   // cells x0 .. x0+3 of row y
    uint32_t d = 0, sw = 0, fl = 0;
    xy2d_levels(x0, y, lg, 2, d, sw, fl);
#pragma unroll
    for (uint32_t j = 0; j < 4; ++j) {   // the last two levels: x bits j
      uint32_t dj = d, swj = sw, flj = fl;
      xy2d_levels(x0 | j, y, 2, 0, dj, swj, flj);
      out[j] = dj;
    }
    store4(job.rank, m, out, vec);
  }
}

// ---------------------------------------------------------------------------
// Four levels per step: lookup tables indexed by the orientation state
// s = sw | fl << 1 and four levels' worth of input, top level first.
//   d2xy[s << 8 | four curve digits]   = x4 | y4 << 4 | s' << 8
//   xy2d[s << 8 | x4 << 4 | y4]        = four curve digits | s' << 8
// (s' = the state after the four levels). Built at compile time by the same
// per-level rules as d2xy_levels / xy2d_levels.
struct HilbertLut {
  uint16_t d2xy[1024];
  uint16_t xy2d[1024];
};

constexpr HilbertLut make_hilbert_lut() {
  HilbertLut t{};
  for (uint32_t s = 0; s < 4; ++s) {
    for (uint32_t dg = 0; dg < 256; ++dg) {
      uint32_t sw = s & 1u, fl = s >> 1, x = 0, y = 0;
      for (int l = 3; l >= 0; --l) {
        const uint32_t q = (dg >> (2 * l)) & 3u;
        const uint32_t a = q >> 1, b = (q ^ a) & 1u, tt = ((a ^ b) & sw) ^ fl;
        x |= (a ^ tt) << l;
        y |= (b ^ tt) << l;
        sw ^= turn_sw(q);
        fl ^= turn_fl(q);
      }
      t.d2xy[s << 8 | dg] = (uint16_t)(x | y << 4 | (sw | fl << 1) << 8);
    }
    for (uint32_t xy = 0; xy < 256; ++xy) {
      const uint32_t x4 = xy >> 4, y4 = xy & 15u;
      uint32_t sw = s & 1u, fl = s >> 1, d = 0;
      for (int l = 3; l >= 0; --l) {
        uint32_t a = ((x4 >> l) & 1u) ^ fl, b = ((y4 >> l) & 1u) ^ fl;
        const uint32_t tt = (a ^ b) & sw;
        a ^= tt;
        b ^= tt;
        const uint32_t q = (a << 1) | (a ^ b);
        d |= q << (2 * l);
        sw ^= turn_sw(q);
        fl ^= turn_fl(q);
      }
      t.xy2d[s << 8 | xy] = (uint16_t)(d | (sw | fl << 1) << 8);
    }
  }
  return t;
}

// ---------------------------------------------------------------------------
// Level-3 blocks: on a curve of side >= 8, the 64 positions 64b .. 64b + 63 are
// one aligned 8 x 8 sub-square, whose cells the curve visits in the order of the
// 3-level curve from the orientation state s entering the block. So the cell of
// position p is the block's origin plus a local cell that depends only on
// (p mod 64, s).
// The local cell (lx | ly << 3) of local position p < 64 in a block entered in
// state st = sw | fl << 1.
constexpr uint32_t hilbert_local_walk(uint32_t p, uint32_t st) {
  uint32_t sw = st & 1u, fl = st >> 1, x = 0, y = 0;
  for (int l = 2; l >= 0; --l) {
    const uint32_t q = (p >> (2 * l)) & 3u;
    const uint32_t a = q >> 1, b = (q ^ a) & 1u, tt = ((a ^ b) & sw) ^ fl;
    x |= (a ^ tt) << l;
    y |= (b ^ tt) << l;
    sw ^= turn_sw(q);
    fl ^= turn_fl(q);
  }
  return x | y << 3;
}

// Entering a block in another state only transposes it (sw) and mirrors both
// coordinates (fl): the local cell for state st from the one for state 0.
constexpr uint32_t hilbert_local_state(uint32_t c0, uint32_t st) {
  const uint32_t c = (st & 1u) ? ((c0 & 7u) << 3 | c0 >> 3) : c0;
  return (st & 2u) ? c ^ 63u : c;
}

constexpr bool hilbert_local_states_agree() {
  for (uint32_t p = 0; p < 64; ++p)
    for (uint32_t st = 0; st < 4; ++st)
      if (hilbert_local_state(hilbert_local_walk(p, 0), st) != hilbert_local_walk(p, st)) return false;
  return true;
}
static_assert(hilbert_local_states_agree(), "block orientations are transposes and mirrors");

// Block b of the 2^lg square (lg >= 3): the cell origin (x, y: bits 3 and up)
// and the state entering the block.
__device__ __forceinline__ void hilbert_block(uint32_t b, int lg, uint32_t &x, uint32_t &y,
                                              uint32_t &st) {
  uint32_t sw = 0, fl = 0;
  x = y = 0;
  d2xy_levels(b << 6, lg, 3, x, y, sw, fl);
  st = sw | fl << 1;
}

// The grid row of a cell given its block origin and its local cell.
__device__ __forceinline__ uint32_t hilbert_block_row(uint32_t bx, uint32_t by, uint32_t cell,
                                                      int lg) {
  return (by | (cell >> 3)) << lg | (bx | (cell & 7u));
}

// Block b of the job with the tables in LDS. A walk of nl levels starts at the
// top of ceil(nl / 4) groups: the padding levels above the curve have digit 0
// and coordinate bits 0, and each of them only toggles sw, so the walk starts
// with sw = (number of padding levels) mod 2.
__device__ __forceinline__ void hilbert4_block_lut(const HilbertJob &job, int32_t b, int32_t tid,
                                                   const HilbertLut &lut) {
  const int32_t lg = job.lg, n4 = job.n4;
  const bool vec = job.vec != 0;
  uint32_t out[4];
  if (b < job.blocks_order) {
    const int32_t m = b * 256 + tid;
    if (m >= n4) return;
    // levels lg-1 .. 1 of d = 4m are levels lg-2 .. 0 of m (a curve of side
    // 2^(lg-1), one level coarser); level 0 is digit j of entry j
    const int nl = lg - 1, ng = (nl + 3) >> 2;
    uint32_t st = (uint32_t)(4 * ng - nl) & 1u, x = 0, y = 0;
    for (int g = ng - 1; g >= 0; --g) {
      const uint32_t e = lut.d2xy[st << 8 | (((uint32_t)m >> (8 * g)) & 255u)];
      x = x << 4 | (e & 15u);
      y = y << 4 | ((e >> 4) & 15u);
      st = e >> 8;
    }
    const uint32_t sw = st & 1u, fl = st >> 1;
#pragma unroll
    for (uint32_t j = 0; j < 4; ++j) {
      const uint32_t a = j >> 1, bb = (j ^ a) & 1u, t = ((a ^ bb) & sw) ^ fl;
      out[j] = ((y << 1 | (bb ^ t)) << lg) | (x << 1 | (a ^ t));
    }
    store4nt(job.order, m, out, vec);
  } else {
    const int32_t m = (b - job.blocks_order) * 256 + tid;
    if (m >= n4) return;
    const uint32_t t0 = 4u * (uint32_t)m;
    const uint32_t y = t0 >> lg, xs = (t0 & ((1u << lg) - 1u)) >> 2, ys = y >> 2;
    // levels lg-1 .. 2 (shared by the four cells x0 .. x0+3 of row y)
    const int nl = lg - 2, ng = (nl + 3) >> 2;
    uint32_t st = (uint32_t)(4 * ng - nl) & 1u, d = 0;
    for (int g = ng - 1; g >= 0; --g) {
      const uint32_t e = lut.xy2d[st << 8 | ((xs >> (4 * g)) & 15u) << 4 | ((ys >> (4 * g)) & 15u)];
      d = d << 8 | (e & 255u);
      st = e >> 8;
    }
    // levels 1, 0 of cell x0 + j: a lookup whose top two levels are padding
    // (two toggles of sw: the state is unchanged)
#pragma unroll
    for (uint32_t j = 0; j < 4; ++j)
      out[j] = d << 4 | (lut.xy2d[st << 8 | j << 4 | (y & 3u)] & 15u);
    store4nt(job.rank, m, out, vec);
  }
}

}  // namespace hla

