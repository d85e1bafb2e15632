// Hilbert index and its inverse (Sec. 3.1-3.2: tokens are reordered along a
// Hilbert curve; the path depends only on (H, W) and is computed once and
// cached).
//
// One launch writes both outputs, coalesced:
//   order[d] = y*W + x of the d-th cell on the curve,
//   rank[t]  = the curve position of cell t = y*W + x.
// Writing rank directly (instead of rank[order[d]] = d) keeps both passes
// coalesced. Both directions walk the curve's levels from the coarsest down,
// carrying the orientation of the current sub-square as two bits: sw (the axes
// are swapped) and fl (both axes are reflected). Curve convention: starts at
// (0,0), first step to (0,1), ends at (side-1, 0); the four quadrants are
// visited lower-left, upper-left, upper-right, lower-right, and the sub-curves
// of the lower-left and lower-right quadrants are the transposed and the
// anti-transposed curve. In (sw, fl) those transforms are (1, 0) and (1, 1) and
// composing them is an xor, so a level costs a few bit operations and no branch.
// Four consecutive positions (or four cells of a row) share every level but the
// last one (two), so each thread walks the shared levels once and writes four
// results with one 16-byte store. On 2^k squares the walk takes four levels per
// step from lookup tables in LDS (the per-level walk cost about 14 vector
// instructions per level and made the kernel vector-bound: 44 -> 25.5 us at
// 4096 x 4096).
//
#include "hilbert_common.h"

namespace hla {
namespace {

// The four-level tables, in constant memory; each workgroup copies them to LDS.
__constant__ HilbertLut kHilbertLut = make_hilbert_lut();
static_assert(sizeof(HilbertLut) == 256 * 16, "one 16-byte copy per thread");

// side = 2^lg >= 4: the workgroups walk the job's 256-thread blocks, grid-strided,
// with the tables in LDS.
__global__ void __launch_bounds__(256) hilbert_square4(HilbertJob job) {
  __shared__ __attribute__((aligned(16))) HilbertLut lut;
  reinterpret_cast<uint4 *>(&lut)[threadIdx.x] = reinterpret_cast<const uint4 *>(&kHilbertLut)[threadIdx.x];
  __syncthreads();
  for (int32_t b = (int32_t)blockIdx.x; b < job.blocks; b += (int32_t)gridDim.x)
    hilbert4_block_lut(job, b, (int32_t)threadIdx.x, lut);
}

// Any side = 2^lg (the small squares, side < 4): one thread per entry.
__global__ void __launch_bounds__(256) hilbert_square1(int32_t lg, int32_t n,
                                                       int32_t *__restrict__ order,
                                                       int32_t *__restrict__ rank) {
  const int32_t i = blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  if (order) {
    uint32_t x = 0, y = 0, sw = 0, fl = 0;
    d2xy_levels((uint32_t)i, lg, 0, x, y, sw, fl);
    order[i] = (int32_t)((y << lg) | x);
  }
  if (rank) {
    uint32_t d = 0, sw = 0, fl = 0;
    xy2d_levels((uint32_t)i & ((1u << lg) - 1u), (uint32_t)i >> lg, lg, 0, d, sw, fl);
    rank[i] = (int32_t)d;
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
  int32_t lg = 0;
  while ((1 << lg) < side) ++lg;
  // position of (cx, cy) on the enclosing side x side curve
  uint32_t d = 0;
  {
    uint32_t sw = 0, fl = 0;
    xy2d_levels((uint32_t)cx, (uint32_t)cy, lg, 0, d, sw, fl);
  }
  // Walk the curve's quadrant tree top-down. The current sub-square's local
  // coordinates p map to grid coordinates P + M p (M a signed permutation).
  // The curve visits quadrants 0..3 at local origins (0,0), (0,s), (s,s), (s,0);
  // quadrant 0 is transposed, quadrant 3 anti-transposed.
  int32_t px = 0, py = 0, m00 = 1, m01 = 0, m10 = 0, m11 = 1;
  uint32_t before = 0;
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
  if (!order && !rank) return hipSuccess;
  int32_t lg = 0;
  while ((1 << lg) < side) ++lg;
  const int32_t n = side * side;
  if (lg < 2) {
    hipLaunchKernelGGL(hilbert_square1, dim3((n + 255) / 256), dim3(256), 0, s, lg, n, order, rank);
    return hipGetLastError();
  }
  const HilbertJob job = make_hilbert_job(lg, order, rank);
  // (eight workgroups per CU at most: each copies the 4 KiB of tables once)
  const int32_t grid = job.blocks < 2048 ? job.blocks : 2048;
  hipLaunchKernelGGL(hilbert_square4, dim3(grid), dim3(256), 0, s, job);
  return hipGetLastError();
}

}  // namespace hla
