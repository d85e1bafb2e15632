// Hilbert index and its inverse (Sec. 3.1-3.2: tokens are reordered along a
// Hilbert curve; the path depends only on (H, W) and is computed once and
// cached).
//
// One launch, one thread per output element, both outputs written coalesced:
//   hilbert_d2xy: thread d walks the curve index two bits per level, from the
//                 finest quadrant up, and writes order[d] = y*W + x;
//   hilbert_xy2d: thread t = y*W + x walks the cell's coordinate bits from the
//                 coarsest level down and writes rank[t] = d.
// Writing rank directly (instead of rank[order[d]] = d) keeps both passes
// coalesced. Curve convention: starts at (0,0), first step to (0,1), ends at
// (side-1, 0); at each level the lower-left quadrant is transposed and the
// lower-right anti-transposed.
//
// Any other H x W grid (the paper also measures 56^2, 96^2, 160^2 and 128 x 256
// grids without saying how its curve covers them): the path is the curve on the
// smallest 2^k square holding the grid, with the cells outside the grid left out
// in the curve's order. hilbert_grid is one thread per grid cell: the cell's
// position d on the enclosing curve, then its rank = the number of grid cells
// the curve visits before d, summed top-down over the curve's levels as the
// areas of grid inside the earlier sibling quadrants - no scan and no scratch
// memory. rank is written coalesced, order scattered (once per grid size).
#include "hla_internal.h"

namespace hla {
namespace {

__device__ __forceinline__ void hilbert_d2xy(int32_t side, int32_t d,
                                             int32_t *__restrict__ order) {
  uint32_t x = 0, y = 0, t = (uint32_t)d;
  for (uint32_t s = 1; s < (uint32_t)side; s <<= 1) {
    // quadrant at this level: 0 lower-left, 1 upper-left, 2 upper-right, 3 lower-right
    const uint32_t qx = (t >> 1) & 1u;          // right half
    const uint32_t qy = (t ^ qx) & 1u;          // upper half
    if (!qy) {                                  // lower quadrants are reflected
      if (qx) {
        x = s - 1 - x;
        y = s - 1 - y;
      }
      const uint32_t tmp = x;
      x = y;
      y = tmp;
    }
    x += s * qx;
    y += s * qy;
    t >>= 2;
  }
  order[d] = (int32_t)(y * (uint32_t)side + x);
}

__device__ __forceinline__ void hilbert_xy2d(int32_t side, int32_t id,
                                             int32_t *__restrict__ rank) {
  uint32_t x = (uint32_t)id % (uint32_t)side;
  uint32_t y = (uint32_t)id / (uint32_t)side;
  uint32_t d = 0;
  for (uint32_t s = (uint32_t)side >> 1; s > 0; s >>= 1) {
    const uint32_t qx = (x & s) ? 1u : 0u;
    const uint32_t qy = (y & s) ? 1u : 0u;
    d += s * s * ((3u * qx) ^ qy);
    if (!qy) {  // undo the reflection of the lower quadrants (only low bits matter below)
      if (qx) {
        x = (s - 1) - (x & (s - 1));
        y = (s - 1) - (y & (s - 1));
      }
      const uint32_t tmp = x;
      x = y;
      y = tmp;
    }
  }
  rank[id] = (int32_t)d;
}

// One launch for both directions: the first `blocks_order` workgroups write order,
// the rest write rank (either part may be absent).
__global__ void __launch_bounds__(256) hilbert_square(int32_t side, int32_t n, int32_t blocks_order,
                                                      int32_t *__restrict__ order,
                                                      int32_t *__restrict__ rank) {
  if ((int32_t)blockIdx.x < blocks_order) {
    const int32_t d = blockIdx.x * 256 + threadIdx.x;
    if (d < n) hilbert_d2xy(side, d, order);
  } else {
    const int32_t id = (blockIdx.x - blocks_order) * 256 + threadIdx.x;
    if (id < n) hilbert_xy2d(side, id, rank);
  }
}

// Cells of the grid [0, W) x [0, H) inside the axis-aligned square spanned by the
// two (opposite) corner points a and b.
__device__ __forceinline__ uint32_t area_inside(int32_t ax, int32_t ay, int32_t bx, int32_t by,
                                                int32_t W, int32_t H) {
  const int32_t x0 = min(ax, bx), x1 = min(max(ax, bx), W - 1);
  const int32_t y0 = min(ay, by), y1 = min(max(ay, by), H - 1);
  return (x1 >= x0 && y1 >= y0) ? (uint32_t)(x1 - x0 + 1) * (uint32_t)(y1 - y0 + 1) : 0u;
}

__global__ void __launch_bounds__(256) hilbert_grid(int32_t H, int32_t W, int32_t side,
                                                    int32_t *__restrict__ order,
                                                    int32_t *__restrict__ rank) {
  const int32_t t = blockIdx.x * 256 + threadIdx.x;
  if (t >= H * W) return;
  const int32_t cx = t % W, cy = t / W;
  // position of (cx, cy) on the enclosing side x side curve
  uint32_t d = 0;
  {
    uint32_t x = (uint32_t)cx, y = (uint32_t)cy;
    for (uint32_t s = (uint32_t)side >> 1; s > 0; s >>= 1) {
      const uint32_t qx = (x & s) ? 1u : 0u;
      const uint32_t qy = (y & s) ? 1u : 0u;
      d += s * s * ((3u * qx) ^ qy);
      if (!qy) {
        if (qx) {
          x = (s - 1) - (x & (s - 1));
          y = (s - 1) - (y & (s - 1));
        }
        const uint32_t tmp = x;
        x = y;
        y = tmp;
      }
    }
  }
  // Walk the curve's quadrant tree top-down. The current sub-square's local
  // coordinates p map to grid coordinates P + M p (M a signed permutation).
  // The curve visits quadrants 0..3 at local origins (0,0), (0,s), (s,s), (s,0);
  // quadrant 0 is transposed, quadrant 3 anti-transposed.
  int32_t px = 0, py = 0, m00 = 1, m01 = 0, m10 = 0, m11 = 1;
  uint32_t before = 0;
  int32_t lg = 0;
  while ((1 << lg) < side) ++lg;
  for (int32_t l = lg - 1; l >= 0; --l) {
    const int32_t s = 1 << l;
    const uint32_t j = (d >> (2 * l)) & 3u;
    const int32_t ox[4] = {0, 0, s, s}, oy[4] = {0, s, s, 0};
    for (uint32_t i = 0; i < j; ++i) {
      const int32_t ax = px + m00 * ox[i] + m01 * oy[i];
      const int32_t ay = py + m10 * ox[i] + m11 * oy[i];
      const int32_t bx = ax + m00 * (s - 1) + m01 * (s - 1);
      const int32_t by = ay + m10 * (s - 1) + m11 * (s - 1);
      before += area_inside(ax, ay, bx, by, W, H);
    }
    // descend: p = o_j + c_j + R_j p'
    int32_t cxo = ox[j], cyo = oy[j];
    if (j == 3) {  // anti-transpose: (u, v) -> (s-1-v, s-1-u)
      cxo += s - 1;
      cyo += s - 1;
    }
    px += m00 * cxo + m01 * cyo;
    py += m10 * cxo + m11 * cyo;
    if (j == 0) {  // transpose: columns of M swap
      const int32_t a = m00, b = m10;
      m00 = m01; m10 = m11; m01 = a; m11 = b;
    } else if (j == 3) {  // anti-transpose: columns swap and change sign
      const int32_t a = m00, b = m10;
      m00 = -m01; m10 = -m11; m01 = -a; m11 = -b;
    }
  }
  if (rank) rank[t] = (int32_t)before;
  if (order) order[before] = t;
}

}  // namespace

hipError_t launch_hilbert_grid(int32_t H, int32_t W, int32_t *order, int32_t *rank,
                               hipStream_t s) {
  int32_t side = 1;
  while (side < H || side < W) side <<= 1;
  const int32_t n = H * W;
  hipLaunchKernelGGL(hilbert_grid, dim3((n + 255) / 256), dim3(256), 0, s, H, W, side, order, rank);
  return hipGetLastError();
}

hipError_t launch_hilbert_perm(int32_t side, int32_t *order, int32_t *rank,
                               hipStream_t s) {
  const int32_t n = side * side;
  const int32_t blocks = (n + 255) / 256;
  const int32_t bo = order ? blocks : 0, br = rank ? blocks : 0;
  if (bo + br == 0) return hipSuccess;
  hipLaunchKernelGGL(hilbert_square, dim3(bo + br), dim3(256), 0, s, side, n, bo, order, rank);
  return hipGetLastError();
}

}  // namespace hla
