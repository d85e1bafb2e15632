// Hilbert index and its inverse on a 2^k x 2^k grid (Sec. 3.1-3.2: tokens are
// reordered along a Hilbert curve; the path depends only on (H, W) and is
// computed once and cached).
//
// Both kernels are one thread per output element and write coalesced:
//   hilbert_d2xy: thread d walks the curve index two bits per level, from the
//                 finest quadrant up, and writes order[d] = y*W + x;
//   hilbert_xy2d: thread t = y*W + x walks the cell's coordinate bits from the
//                 coarsest level down and writes rank[t] = d.
// Writing rank directly (instead of rank[order[d]] = d) keeps both passes
// coalesced. Curve convention: starts at (0,0), first step to (0,1), ends at
// (side-1, 0); at each level the lower-left quadrant is transposed and the
// lower-right anti-transposed.
#include "hla_internal.h"

namespace hla {
namespace {

__global__ void __launch_bounds__(256) hilbert_d2xy(int32_t side, int32_t n,
                                                    int32_t *__restrict__ order) {
  const int32_t d = blockIdx.x * 256 + threadIdx.x;
  if (d >= n) return;
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

__global__ void __launch_bounds__(256) hilbert_xy2d(int32_t side, int32_t n,
                                                    int32_t *__restrict__ rank) {
  const int32_t id = blockIdx.x * 256 + threadIdx.x;
  if (id >= n) return;
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

}  // namespace

hipError_t launch_hilbert_perm(int32_t side, int32_t *order, int32_t *rank,
                               hipStream_t s) {
  const int32_t n = side * side;
  const int32_t blocks = (n + 255) / 256;
  if (order) {
    hipLaunchKernelGGL(hilbert_d2xy, dim3(blocks), dim3(256), 0, s, side, n, order);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (rank) {
    hipLaunchKernelGGL(hilbert_xy2d, dim3(blocks), dim3(256), 0, s, side, n, rank);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace hla
