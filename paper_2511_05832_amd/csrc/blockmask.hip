// Tile classification and per-row / per-column tile lists (Sec. 3.1: full, partial and
// empty blocks of the N x N score matrix; empty blocks are skipped, full
// blocks run without a mask, partial blocks need the element mask).
//
// Exact closed-form classification (tiles_common.h), one thread per (query
// tile, key tile).
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
#include "tiles_common.h"

namespace hla {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

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
      cls = tile_class(p, tile_m, tile_n, qt, kt);
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
