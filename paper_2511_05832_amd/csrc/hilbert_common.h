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
__device__ __forceinline__ uint32_t turn_sw(uint32_t q) { return 1u ^ ((q ^ (q >> 1)) & 1u); }
__device__ __forceinline__ uint32_t turn_fl(uint32_t q) { return q & (q >> 1) & 1u; }

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

}  // namespace hla

