// Internal declarations shared by the HIP kernels and the C-ABI layer of libhla.
// Launchers assume their arguments were validated by the C-ABI layer and return
// the HIP status of the launch.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hla.h"

namespace hla {

// Exact unsigned division by a runtime constant for numerators below 2^31
// (round-up multiply-high method; Granlund & Montgomery, "Division by invariant
// integers using multiplication", 1994): q = (umulhi(n, mul) + n) >> shift.
struct FastDiv {
  uint32_t div, mul, shift;
};

inline FastDiv make_fastdiv(uint32_t d) {
  FastDiv f;
  f.div = d;
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  f.shift = l;
  f.mul = (uint32_t)(((1ull << 32) * ((1ull << l) - d)) / d + 1);
  return f;
}

__device__ __forceinline__ uint32_t fdiv(uint32_t n, const FastDiv &f) {
  return (__umulhi(n, f.mul) + n) >> f.shift;
}

// Pattern in the form the kernels use. For the 1-D (Hilbert) patterns every
// query's allowed keys form one interval [lo, hi]; for the 2-D row-major
// patterns they form one rectangle of grid cells. See query_interval() and
// query_rect() in the kernels.
struct PatternArgs {
  int32_t kind;
  int32_t H, W, N;
  int32_t p0, p1;
  FastDiv wdiv;  // division by W (row-major patterns)
};

inline bool pattern_is_1d(int32_t kind) {
  return kind == HLA_HILBERT_WINDOW || kind == HLA_HILBERT_SLIDE ||
         kind == HLA_HILBERT_NEIGHBORHOOD || kind == HLA_HILBERT_SHIFTED_WINDOW;
}

// Compute units of the current device, read once per device (256 if the query
// fails).
inline int device_cu_count() {
  static int cus_of[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cus_of[dev]) {
    int n = 0;
    cus_of[dev] =
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0 ? n : 256;
  }
  return cus_of[dev];
}

inline PatternArgs make_pattern_args(const hla_pattern_desc &p) {
  PatternArgs a;
  a.kind = p.pattern;
  a.H = p.H;
  a.W = p.W;
  a.N = p.H * p.W;
  a.p0 = p.p0;
  a.p1 = p.p1;
  a.wdiv = make_fastdiv((uint32_t)p.W);
  return a;
}

hipError_t launch_hilbert_perm(int32_t side, int32_t *order, int32_t *rank,
                               hipStream_t s);
// Any H x W grid: the enclosing 2^k curve with the cells outside the grid left out.
hipError_t launch_hilbert_grid(int32_t H, int32_t W, int32_t *order, int32_t *rank,
                               hipStream_t s);

hipError_t launch_permute(const void *src, void *dst, const int32_t *order,
                          int64_t BH, int64_t N, int64_t row_bytes, bool scatter,
                          hipStream_t s);

// One direction of tile lists: per line, the count and ascending -1-padded list
// of the full tiles and of the partial tiles.
struct BlockLists {
  int32_t *n_full, *full_idx, *n_part, *part_idx;
};

struct HilbertJob;

// Row lists always; column lists when cols is not NULL; totals (of the row
// lists) when totals is not NULL. path (optional): a Hilbert index job run by
// extra workgroups of the row-list launch.
hipError_t launch_block_mask(const PatternArgs &pat, int32_t tile_m,
                             int32_t tile_n, int32_t n_qtiles, int32_t n_ktiles,
                             const BlockLists &rows, const BlockLists *cols,
                             int32_t *totals, hipStream_t s, const HilbertJob *path = nullptr);

// The Hilbert index of a side x side square (side a power of two >= 4) and the
// tile lists in one launch (plus the column-list and totals launches if asked).
hipError_t launch_path_and_mask(int32_t side, int32_t *order, int32_t *rank,
                                const PatternArgs &pat, int32_t tile_m, int32_t tile_n,
                                int32_t n_qtiles, int32_t n_ktiles, const BlockLists &rows,
                                const BlockLists *cols, int32_t *totals, hipStream_t s);

// Forward modes: plain (tensors in sequence order), gather (tensors in grid
// order, sequence position i is row order[i]), rpb (tensors in sequence order,
// plus the global relative position bias looked up from the grid cells order[i]),
// hilbert (as gather, with the rows taken from the Hilbert curve of the 2^lg
// square and the tile lists classified inside the kernel: no order array, no
// lists).
enum AttnMode { ATTN_PLAIN = 0, ATTN_GATHER = 1, ATTN_RPB = 2, ATTN_HILBERT = 3 };

struct AttnArgs {
  const void *q, *k, *v;
  void *out;
  float *lse;
  const int32_t *order;  // grid row of each sequence position (gather, rpb), else NULL
  const float *rpb;      // rpb: [heads, 2H-1, 2W-1] bias table, else NULL
  int32_t mode;          // AttnMode
  const int32_t *n_full, *full_idx, *n_part, *part_idx;
  int32_t BH, heads, N, n_qtiles, n_ktiles;
  float scale, scale_log2;  // scale, scale * log2(e)
  PatternArgs pat;
  int32_t lg;               // hilbert: log2 of the grid side (N = 4^lg)
  int32_t hgroups;          // hilbert: groups the B * heads slices are split into (else BH)
};

hipError_t launch_attn_bf16(const AttnArgs &a, int d, int tile_m, int tile_n,
                            hipStream_t s);
hipError_t launch_attn_f32(const AttnArgs &a, int d, int tile_m, int tile_n,
                           hipStream_t s);

struct AttnBwdArgs {
  const void *q, *k, *v, *out, *dout;
  const float *lse;
  float *stats;  // per row: (lse * log2 e, -delta), 2 floats
  void *dq, *dk, *dv;
  // Fused reordering: every tensor (and lse, stats) stored in grid order, and
  // sequence position i is row order[i]; NULL: tensors in sequence order.
  const int32_t *order;
  const int32_t *n_full, *full_idx, *n_part, *part_idx;          // per query-tile row
  const int32_t *n_full_t, *full_idx_t, *n_part_t, *part_idx_t;  // per key-tile column
  int32_t BH, N, n_qtiles, n_ktiles;
  float scale, scale_log2;
  PatternArgs pat;
  // The heads split into hgroups near-equal groups of consecutive heads, one
  // group per workgroup and tile (set by each kernel's launcher; BH: one head)
  int32_t hgroups;
};


// Row statistics, then the query gradients (row lists), then the key and value
// gradients (column lists), all on stream s.
hipError_t launch_attn_bwd_bf16(const AttnBwdArgs &a, int d, int tile_m, int tile_n,
                                hipStream_t s);
hipError_t launch_attn_bwd_f32(const AttnBwdArgs &a, int d, int tile_m, int tile_n,
                               hipStream_t s);

// order: null, or the reordering fused in (QKV reads x row b*N + order[n],
// the output projection writes y row b*N + order[n]).
hipError_t launch_qkv_proj(const void *x, const void *w, const int32_t *order, void *q, void *k,
                           void *v, int64_t B, int64_t N, int64_t heads, int64_t d,
                           hipStream_t s);
hipError_t launch_out_proj(const void *o, const void *w, const int32_t *order, void *y, int64_t B,
                           int64_t N, int64_t heads, int64_t d, int64_t c_out, hipStream_t s);

}  // namespace hla
