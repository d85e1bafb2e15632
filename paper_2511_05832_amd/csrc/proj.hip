// Token-wise linear projections of the layer pipeline, with the head split /
// merge folded into the addressing (Sec. 4.2, input processing: the QKV
// projection follows the Hilbert reordering; Sec. 3.3: the attention output is
// projected back).
//
//   QKV:  y[t, f] = sum_k x[t, k] W[f, k], f in [0, 3C), scattered into
//         q / k / v [B, heads, N, d] by f -> (which, head, e)
//   out:  y[t, f] = sum_k o[b, k/d, n, k%d] W[f, k]  (heads merged on the fly)
//
// MFMA D = A B with A = a tile of W (features x k), B = the input rows (k x
// tokens), v_mfma_f32_32x32x16_bf16, fp32 accumulation. A workgroup of four
// waves handles FT features of a group of blocks of 128 tokens: the FT x K weight
// tile sits in LDS (padded rows) for all of them, and each wave streams the
// K-slices of its own 32 tokens of a block straight from global memory (16
// contiguous bytes per lane per step). The accumulator lane layout gives each
// lane one token and runs of four consecutive features, stored as 8-byte bf16
// writes.
//
// Grid. A 1-D grid in which the workgroups of one token group (all its feature
// tiles) get the same blockIdx.x % 8, i.e. the same XCD (workgroups are dealt
// round-robin to the 8 XCDs), and neighbouring ids, so the input rows that every
// feature tile reads come from that XCD's L2 after the first read instead of
// from HBM once per feature tile.
#include "attn_common.h"

namespace hla {
namespace {

constexpr int kWaves = 4;
constexpr int kTokens = 32 * kWaves;
constexpr int kXcds = 8;

struct ProjArgs {
  const __bf16 *in;   // x [T, K] (QKV) or o [B, heads, N, d] (out)
  // null, or the reordering fused in: QKV reads token n of batch b from input
  // row b*N + order[n]; the output projection writes it to row b*N + order[n]
  const int32_t *order;
  const __bf16 *w;    // [F, K]
  __bf16 *out0, *out1, *out2;  // q, k, v (QKV) or y (out, out0 only)
  int32_t T, N, K, F, heads, d, C;
  int32_t n_ftiles, group, n_groups;  // feature tiles; token blocks per group; groups
};

// MODE 0: QKV (head split on output). MODE 1: out projection (head merge on input).
template <int FB, int MODE>
__global__ void __launch_bounds__(64 * kWaves) proj_kernel(ProjArgs p) {
  constexpr int FT = 32 * FB;
  extern __shared__ __attribute__((aligned(16))) __bf16 wl[];
  const int WS = p.K + 8;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, half = lane >> 5;
  // (token group, feature tile) of this workgroup: id L = 8 s + x goes to XCD x;
  // its s-th slot there is feature tile s % n_ftiles of token group
  // (s / n_ftiles) * 8 + x. The grid covers a multiple of 8 token groups, the
  // surplus ones return here.
  const int xcd = blockIdx.x % kXcds, s = blockIdx.x / kXcds;
  const int group = (s / p.n_ftiles) * kXcds + xcd;
  if (group >= p.n_groups) return;
  const int fbase = (s % p.n_ftiles) * FT;

  // weight tile -> LDS
  const int cpr = p.K / 8;
  for (int i = tid; i < FT * cpr; i += 64 * kWaves) {
    const int r = i / cpr, c = i - r * cpr;
    *reinterpret_cast<uint4 *>(wl + r * WS + c * 8) =
        *reinterpret_cast<const uint4 *>(p.w + (int64_t)(fbase + r) * p.K + c * 8);
  }
  __syncthreads();

  for (int blk = group * p.group; blk < group * p.group + p.group; ++blk) {
  const int t = blk * kTokens + wave * 32 + col;
  if (blk * kTokens >= p.T) break;
  const bool valid = t < p.T;
  const int tt = valid ? t : 0;
  const int b = tt / p.N, n = tt - b * p.N;

  f32x16 acc[FB];
#pragma unroll
  for (int f = 0; f < FB; ++f) acc[f] = f32x16{};

  for (int k0 = 0; k0 < p.K; k0 += 64) {
    bf16x8 xin[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int k = k0 + 16 * c + 8 * half;
      const __bf16 *src;
      if (MODE == 0) {
        src = p.in + (p.order ? (int64_t)b * p.N + p.order[n] : (int64_t)tt) * p.K + k;
      } else {
        const int h = k / p.d, e = k - h * p.d;
        src = p.in + ((int64_t)(b * p.heads + h) * p.N + n) * p.d + e;
      }
      xin[c] = *reinterpret_cast<const bf16x8 *>(src);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
#pragma unroll
      for (int f = 0; f < FB; ++f) {
        const bf16x8 wop =
            *reinterpret_cast<const bf16x8 *>(wl + (f * 32 + col) * WS + k0 + 16 * c + 8 * half);
        acc[f] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wop, xin[c], acc[f], 0, 0, 0);
      }
    }
  }

  if (!valid) continue;
#pragma unroll
  for (int f = 0; f < FB; ++f) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int feat = fbase + f * 32 + 8 * g + 4 * half;
      bf16x4 o4;
#pragma unroll
      for (int j = 0; j < 4; ++j) o4[j] = (__bf16)acc[f][4 * g + j];
      __bf16 *dst;
      if (MODE == 0) {
        const int which = feat / p.C, r = feat - which * p.C;
        const int h = r / p.d, e = r - h * p.d;
        __bf16 *base = which == 0 ? p.out0 : (which == 1 ? p.out1 : p.out2);
        dst = base + ((int64_t)(b * p.heads + h) * p.N + n) * p.d + e;
      } else {
        dst = p.out0 + (p.order ? (int64_t)b * p.N + p.order[n] : (int64_t)tt) * p.F + feat;
      }
      *reinterpret_cast<bf16x4 *>(dst) = o4;
    }
  }
  }
}

// Rows-resident variant (K = 16 KC <= 192): one workgroup per block of 128
// tokens holds its rows' K-slices in registers (read from HBM once) and walks
// every feature tile, each tile's weights copied from L2 into one of two LDS
// buffers with the 16-byte LDS DMA while the previous tile is multiplied. Per
// tile j: issue tile j + 1's copies, then the stores of tile j - 1 (kept in
// registers as bf16), then the products, then a wait that leaves exactly those
// stores in flight (the vmcnt counter is in order, so the older copies must have
// landed) and a barrier (every wave is done with tile j's buffer). Stores never
// hold up a wait. A lane past the last token computes and stores row T - 1 again
// (the same bytes to the same place), so every wave issues the same number of
// stores per tile.
template <int KC, int FB, int MODE>
__global__ void __launch_bounds__(64 * kWaves, 2) proj_rows_kernel(ProjArgs p) {
  constexpr int K = 16 * KC;
  constexpr int FT = 32 * FB;
  constexpr int WS = K + 8;                              // padded LDS row, elements
  constexpr int TILE_BUF = (FT * WS * 2 + 1023) / 1024 * 1024;
  constexpr int NCOPY = TILE_BUF / 1024;                 // 1 KiB copies per tile
  __shared__ __attribute__((aligned(16))) char wl[2 * TILE_BUF];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, half = lane >> 5;

  // Copy instruction i of a tile fills LDS bytes [1024 i, 1024 i + 1024) of its
  // buffer, lane l the 16 bytes at o = 1024 i + 16 l: row o / (2 WS), element
  // (o % (2 WS)) / 2. Row padding and the slots past the last row copy a chunk
  // of the weights that nothing reads.
  auto issue_w = [&](int j, int buf) {
    const int fbase = j * FT;
    for (int i = wave; i < NCOPY; i += kWaves) {
      const int o = 1024 * i + 16 * lane;
      int r = o / (2 * WS), e = (o - r * 2 * WS) / 2;
      if (r >= FT) r = FT - 1;
      if (e >= K) e = 0;
      lds_dma16(p.w + (int64_t)(fbase + r) * K + e, lds_addr(wl + buf * TILE_BUF + 1024 * i));
    }
  };

  const int t = blockIdx.x * kTokens + wave * 32 + col;
  const int tt = t < p.T ? t : p.T - 1;
  const int b = tt / p.N, n = tt - b * p.N;
  const int ntiles = p.F / FT;
  constexpr int NST = 4 * FB;   // stores per lane and tile (8 bytes each)
  // Output projection: this token's output row, loaded once, before the loop (a
  // load of the order entry beside the stores made the compiler wait for every
  // copy in flight on each tile).
  int64_t yrow = (int64_t)tt;
  if (MODE == 1 && p.order) yrow = (int64_t)b * p.N + p.order[n];

  // The stores of tile j from its bf16 results (4 consecutive features each).
  // QKV: a 32-feature block lies in one head of one of q, k, v (d % 32 == 0), so
  // its base is wave-uniform and each lane adds a 32-bit element offset (the
  // launcher checks that the outputs fit). Stores then share one uniform base
  // instead of a 64-bit address per store.
  auto store_tile = [&](int j, const bf16x4 (&o)[NST]) {
#pragma unroll
    for (int f = 0; f < FB; ++f) {
      if (MODE == 0) {
        const int f0 = j * FT + f * 32;
        const int which = f0 / p.C, r0 = f0 - which * p.C;
        const int h = r0 / p.d, e0 = r0 - h * p.d;
        __bf16 *base = which == 0 ? p.out0 : (which == 1 ? p.out1 : p.out2);
        const uint32_t row = (uint32_t)((b * p.heads + h) * p.N + n) * (uint32_t)p.d + (uint32_t)e0;
#pragma unroll
        for (int g = 0; g < 4; ++g)
          *reinterpret_cast<bf16x4 *>(base + (row + 8 * g + 4 * half)) = o[4 * f + g];
      } else {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int feat = j * FT + f * 32 + 8 * g + 4 * half;
          *reinterpret_cast<bf16x4 *>(p.out0 + yrow * p.F + feat) = o[4 * f + g];
        }
      }
    }
  };

  issue_w(0, 0);
  bf16x8 xin[KC];
#pragma unroll
  for (int c = 0; c < KC; ++c) {
    const int k = 16 * c + 8 * half;
    const __bf16 *src;
    if (MODE == 0) {
      src = p.in + (p.order ? (int64_t)b * p.N + p.order[n] : (int64_t)tt) * K + k;
    } else {
      const int h = k / p.d, e = k - h * p.d;
      src = p.in + ((int64_t)(b * p.heads + h) * p.N + n) * p.d + e;
    }
    xin[c] = *reinterpret_cast<const bf16x8 *>(src);
  }
  wait_vmem_all();
  wait_then_barrier<0>();

  bf16x4 pend[NST];
  for (int j = 0; j < ntiles; ++j) {
    if (j + 1 < ntiles) issue_w(j + 1, (j + 1) & 1);
    if (j > 0) store_tile(j - 1, pend);
    const __bf16 *wt = reinterpret_cast<const __bf16 *>(wl + (j & 1) * TILE_BUF);
    f32x16 acc[FB];
#pragma unroll
    for (int f = 0; f < FB; ++f) acc[f] = f32x16{};
#pragma unroll
    for (int c = 0; c < KC; ++c)
#pragma unroll
      for (int f = 0; f < FB; ++f) {
        const bf16x8 wop = *reinterpret_cast<const bf16x8 *>(wt + (f * 32 + col) * WS + 16 * c + 8 * half);
        acc[f] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wop, xin[c], acc[f], 0, 0, 0);
      }
#pragma unroll
    for (int f = 0; f < FB; ++f)
#pragma unroll
      for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int q = 0; q < 4; ++q) pend[4 * f + g][q] = (__bf16)acc[f][4 * g + q];
    if (j > 0) wait_then_barrier<NST>();
    else wait_then_barrier<0>();
  }
  store_tile(ntiles - 1, pend);
}

// ---------------------------------------------------------------------------
// Streaming kernel (weights in registers). For the layer's shapes (K = 192,
// F = 576 or 192) the whole weight matrix fits the registers of one workgroup
// of twelve waves: wave w keeps the A operands of its FBW blocks of 16 output
// features for all of K (v_mfma_f32_16x16x32_bf16; FBW * K/32 * 4 VGPRs). The
// workgroup is persistent (one per CU) and streams tiles of 32 tokens:
//  - x rows come into a 5-stage LDS ring by the 16-byte LDS DMA, 1 KiB per
//    instruction, four tiles ahead; the 16-byte chunks of a row are stored XOR-
//    swizzled by (row & 7) (each lane fetches the chunk that belongs in its
//    slot), which puts the B-operand reads (16 rows x one chunk per 16 lanes) on
//    distinct banks;
//  - the results are staged through LDS as [token][feature] rows and written
//    back with non-temporal 16-byte stores in output order: one wave instruction covers 1 KiB
//    of q / k / v (d = 32: 16 consecutive token rows of one head) or of y. (The
//    accumulator layout - four features of one token per lane - stored
//    directly gave 8-byte stores into 32 different rows per instruction and ran
//    at a third of the write bandwidth.)
// Every wave issues the same number of copies and stores per tile (lanes past
// the last token re-read and re-store row T - 1, the same bytes to the same
// place), so each wait leaves an exact number of them in flight: the vmcnt
// counter is in order. With the reordering fused in, the order entries of all
// of the workgroup's tokens are copied into LDS once, before the tiles.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kStreamTT = 32;      // tokens per tile
constexpr int kStreamAhead = 4;    // x tiles in flight ahead of the current one
constexpr int kStreamRing = kStreamAhead + 1;
constexpr int kStreamMaxTiles = 64;  // tiles per workgroup (order entries in LDS)
constexpr int kStreamWaves = 12;

struct StreamArgs {
  const __bf16 *in;        // x [T, K] (QKV) or o [B, heads, N, d] (out)
  const int32_t *order;    // null, or the token reordering fused in (see ProjArgs)
  const __bf16 *w;         // [F, K]
  __bf16 *out0, *out1, *out2;
  int32_t T, N, ntiles;
  FastDiv ndiv;            // division by N
};

// LDS writes of this wave done, then barrier (vector memory left in flight).
__device__ __forceinline__ void lds_then_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// KS = K / 32; D head dim; FBW 16-feature blocks per wave; MODE 0 QKV, 1 output
// projection; ORD: an order array is given.
template <int KS, int D, int FBW, int MODE, bool ORD>
__global__ void __launch_bounds__(64 * kStreamWaves, 1) proj_stream_kernel(StreamArgs p) {
  constexpr int NWV = kStreamWaves;
  constexpr int TT = kStreamTT;
  constexpr int A = kStreamAhead;
  constexpr int R = kStreamRing;
  constexpr int K = 32 * KS;
  constexpr int HEADS = K / D;
  constexpr int F = 16 * FBW * NWV;
  constexpr int CPR = K / 8;                        // 16-byte chunks per x row
  constexpr int XTILE = TT * K * 2;                 // bytes of one x tile
  constexpr int CPW = TT * CPR / (64 * NWV);        // x copies per wave and tile
  constexpr int FP = F + 8;                         // staging row pitch, elements
  constexpr int SPW = TT * F / 8 / (64 * NWV);      // 16-byte stores per wave and tile
  constexpr int XR = 0;
  constexpr int ST = XR + R * XTILE;
  constexpr int IX = ST + TT * FP * 2;
  constexpr int LDSB = IX + (ORD ? kStreamMaxTiles * TT * 4 : 0);
  constexpr int MAXN = CPW * (A - 1) + SPW * A;
  static_assert(TT * CPR % (64 * NWV) == 0 && TT * F / 8 % (64 * NWV) == 0, "work must split evenly");
  static_assert(MODE == 0 ? F == 3 * K : true, "QKV: F = 3 C");
  static_assert(CPR % 8 == 0, "the chunk swizzle works within octets");
  static_assert(MAXN < 64, "vmcnt range");

  __shared__ __attribute__((aligned(16))) char lds[LDSB];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, g4 = lane >> 4;
  const int fw = wave * FBW * 16;   // this wave's first feature

  // Tiles of this workgroup: blockIdx.x, blockIdx.x + gridDim.x, ... (at most
  // kStreamMaxTiles; the launcher sizes the grid for that).
  const int nt = ((int)blockIdx.x < p.ntiles)
                     ? (p.ntiles - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x
                     : 0;
  auto tile_of = [&](int i) { return (int)blockIdx.x + i * (int)gridDim.x; };
  auto clamp_t = [&](int t) { return t < p.T ? t : p.T - 1; };

  // x tile i into ring stage i % R: slot q of the tile holds row q / CPR, chunk
  // (q % CPR) ^ (row & 7) of the source. QKV with an order: entry r of `rows`
  // is the order entry of the tile's token r (`rows` = the LDS copy of the
  // order entries, or, for the first tiles, registers - see below).
  const int32_t *idx_all = reinterpret_cast<const int32_t *>(lds + IX);
  auto issue_x_from = [&](int i, auto row_of) {
    char *stage = lds + XR + (i % R) * XTILE;
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
      const int q = (j * NWV + wave) * 64 + lane;
      const int r = q / CPR, c = (q % CPR) ^ (r & 7);
      const int t = clamp_t(tile_of(i) * TT + r);
      const int b = (int)fdiv((uint32_t)t, p.ndiv), n = t - b * p.N;
      const __bf16 *src;
      if constexpr (MODE == 0) {
        const int64_t row = ORD ? (int64_t)b * p.N + row_of(j, r) : (int64_t)t;
        src = p.in + row * K + 8 * c;
      } else {
        const int h = (8 * c) / D, e = (8 * c) % D;
        src = p.in + ((int64_t)(b * HEADS + h) * p.N + n) * D + e;
      }
      lds_dma16(src, lds_addr(stage + (j * NWV + wave) * 1024));
    }
  };
  auto issue_x = [&](int i) {
    const int32_t *idx = idx_all + i * TT;
    issue_x_from(i, [&](int, int r) { return idx[r]; });
  };

  // Prologue, all in flight together: (QKV with an order) this lane's order
  // entries for the first A tiles, loaded into registers first; the weights (the
  // A operand of block fb, k-step s = W[fw + 16 fb + l16][32 s + 8 g4 ..]); the
  // order entries of every token of this workgroup's tiles into LDS (entry e =
  // token e % 32 of tile e / 32); the x copies of the first A tiles. Then one
  // wait and a barrier. (The compiler's own wait before the first tiles' x
  // addresses covers only the order loads issued ahead of the weights.)
  int first_rows[A][CPW];
  if constexpr (ORD && MODE == 0) {
#pragma unroll
    for (int i = 0; i < A; ++i)
#pragma unroll
      for (int j = 0; j < CPW; ++j) {
        const int r = ((j * NWV + wave) * 64 + lane) / CPR;
        const int t = clamp_t(min(tile_of(i), p.ntiles - 1) * TT + r);
        const int b = (int)fdiv((uint32_t)t, p.ndiv);
        first_rows[i][j] = p.order[t - b * p.N];
      }
  }
  bf16x8 wr[FBW][KS];
#pragma unroll
  for (int fb = 0; fb < FBW; ++fb)
#pragma unroll
    for (int s = 0; s < KS; ++s)
      wr[fb][s] = *reinterpret_cast<const bf16x8 *>(p.w + (int64_t)(fw + 16 * fb + l16) * K + 32 * s + 8 * g4);
  if constexpr (ORD) {
    for (int c = wave; c * 64 < nt * TT; c += NWV) {
      const int e = min(c * 64 + lane, nt * TT - 1);
      const int t = clamp_t(tile_of(e / TT) * TT + e % TT);
      const int b = (int)fdiv((uint32_t)t, p.ndiv);
      lds_dma4(p.order + (t - b * p.N), lds_addr(lds + IX + c * 256));
    }
  }
#pragma unroll
  for (int i = 0; i < A; ++i)
    if (i < nt) issue_x_from(i, [&](int j, int) { return first_rows[i][j]; });
  wait_vmem_all();
  wait_then_barrier<0>();

  // B-operand byte offsets within a stage: token block tb, k-step s.
  int boff[2][KS];
#pragma unroll
  for (int tb = 0; tb < 2; ++tb)
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int r = 16 * tb + l16, c = (4 * s + g4) ^ (r & 7);
      boff[tb][s] = r * K * 2 + c * 16;
    }

  for (int i = 0; i < nt; ++i) {
    // This wave's operations issued after tile i's x copies: the copies of tiles
    // i + 1 .. i + A - 1 and the stores of tiles i - A .. i - 1 (those that exist).
    wait_n_then_barrier<MAXN>(CPW * min(A - 1, nt - 1 - i) + SPW * min(i, A));
    // (stage (i + A) % R held tile i - 1, which every wave finished before the
    // barrier above)
    if (i + A < nt) issue_x(i + A);

    const char *stage = lds + XR + (i % R) * XTILE;
    f32x4 acc[FBW][2];
#pragma unroll
    for (int fb = 0; fb < FBW; ++fb) acc[fb][0] = acc[fb][1] = f32x4{};
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        const bf16x8 xop = *reinterpret_cast<const bf16x8 *>(stage + boff[tb][s]);
#pragma unroll
        for (int fb = 0; fb < FBW; ++fb)
          acc[fb][tb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wr[fb][s], xop, acc[fb][tb], 0, 0, 0);
      }
    // Stage as [token][feature]: lane (l16, g4) of block (fb, tb) holds token
    // 16 tb + l16, features fw + 16 fb + 4 g4 + 0..3. (The staging area was last
    // read in tile i - 1's stores, before the barrier above.)
#pragma unroll
    for (int fb = 0; fb < FBW; ++fb)
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        bf16x4 o4;
#pragma unroll
        for (int e = 0; e < 4; ++e) o4[e] = (__bf16)acc[fb][tb][e];
        *reinterpret_cast<bf16x4 *>(lds + ST + ((16 * tb + l16) * FP + fw + 16 * fb + 4 * g4) * 2) = o4;
      }
    lds_then_barrier();
    // Stores in output order, 16 bytes per lane.
    const int32_t *idx = idx_all + i * TT;
#pragma unroll
    for (int j = 0; j < SPW; ++j) {
      const int q = (j * NWV + wave) * 64 + lane;
      int r, feat;
      __bf16 *dst;
      if constexpr (MODE == 0) {
        // q -> (block = which * heads + h, token r, 8-feature chunk e8), e8 fastest
        constexpr int E8 = D / 8;
        const int e8 = q % E8;
        r = (q / E8) % TT;
        const int blk = q / (E8 * TT);
        feat = blk * D + 8 * e8;
        const int which = blk / HEADS, h = blk % HEADS;
        const int t = clamp_t(tile_of(i) * TT + r);
        const int b = (int)fdiv((uint32_t)t, p.ndiv), n = t - b * p.N;
        __bf16 *base = which == 0 ? p.out0 : (which == 1 ? p.out1 : p.out2);
        dst = base + ((int64_t)(b * HEADS + h) * p.N + n) * D + 8 * e8;
      } else {
        constexpr int CF = F / 8;
        const int c = q % CF;
        r = q / CF;
        feat = 8 * c;
        const int t = clamp_t(tile_of(i) * TT + r);
        const int b = (int)fdiv((uint32_t)t, p.ndiv), n = t - b * p.N;
        const int64_t row = (int64_t)b * p.N + (ORD ? idx[r] : n);
        dst = p.out0 + row * F + feat;
      }
      // non-temporal: the output streams past the caches (measured 13% faster
      // for the QKV projection, and the attention reading q, k, v next no slower)
      const u32x4 v = *reinterpret_cast<const u32x4 *>(lds + ST + (r * FP + feat) * 2);
      __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(dst));
    }
  }
}

template <int D, int MODE, bool ORD>
hipError_t launch_stream(const ProjArgs &a, hipStream_t s) {
  StreamArgs p;
  p.in = a.in;
  p.order = a.order;
  p.w = a.w;
  p.out0 = a.out0;
  p.out1 = a.out1;
  p.out2 = a.out2;
  p.T = a.T;
  p.N = a.N;
  p.ntiles = (a.T + kStreamTT - 1) / kStreamTT;
  p.ndiv = make_fastdiv((uint32_t)a.N);
  int cus = 0, dev = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  // one workgroup per CU, more when a workgroup would get over kStreamMaxTiles tiles
  int grid = p.ntiles < cus ? p.ntiles : cus;
  const int need = (p.ntiles + kStreamMaxTiles - 1) / kStreamMaxTiles;
  if (need > grid) grid = need;
  // QKV: F = 576 = 12 waves x 3 blocks; output projection: F = 192 = 12 waves x 1
  constexpr int FBW = MODE == 0 ? 3 : 1;
  hipLaunchKernelGGL((proj_stream_kernel<6, D, FBW, MODE, ORD>), dim3(grid), dim3(64 * kStreamWaves), 0, s, p);
  return hipGetLastError();
}

template <int MODE>
hipError_t launch_stream_any(const ProjArgs &p, hipStream_t s) {
  if (p.d == 32) return p.order ? launch_stream<32, MODE, true>(p, s) : launch_stream<32, MODE, false>(p, s);
  return p.order ? launch_stream<64, MODE, true>(p, s) : launch_stream<64, MODE, false>(p, s);
}

template <int KC, int MODE>
hipError_t launch_rows(const ProjArgs &p, hipStream_t s) {
  const uint32_t gx = (uint32_t)((p.T + kTokens - 1) / kTokens);
  hipLaunchKernelGGL((proj_rows_kernel<KC, 3, MODE>), dim3(gx), dim3(64 * kWaves), 0, s, p);
  return hipGetLastError();
}

template <int MODE>
hipError_t launch_fb(ProjArgs p, hipStream_t s) {
  // streaming kernel (weights in registers) for K = 192 with F = 576 (QKV) or
  // F = 192 (output projection), d = 32 or 64
  if (p.K == 192 && (p.d == 32 || p.d == 64) && (MODE == 0 ? p.F == 576 : p.F == 192))
    return launch_stream_any<MODE>(p, s);
  // rows-resident kernel where it applies: 96-feature tiles, K = 64, 128 or 192,
  // heads of a multiple of 32 channels, outputs addressable with 32-bit offsets
  if (p.F % 96 == 0 && p.d % 32 == 0 && (int64_t)p.T * p.F < ((int64_t)1 << 31)) {
    if (p.K == 192) return launch_rows<12, MODE>(p, s);
    if (p.K == 128) return launch_rows<8, MODE>(p, s);
    if (p.K == 64) return launch_rows<4, MODE>(p, s);
  }
  const int64_t blocks = (p.T + kTokens - 1) / kTokens;
  // widest feature tile whose weight slice fits the 64 KiB of LDS a workgroup
  // gets without opting in to more
  int fb = 1;
  for (int cand : {6, 3, 2}) {
    if (p.F % (32 * cand) == 0 && (int64_t)32 * cand * (p.K + 8) * 2 <= 64 * 1024) {
      fb = cand;
      break;
    }
  }
  p.n_ftiles = p.F / (32 * fb);
  // token blocks per workgroup (sharing one weight tile): the most of 4, 2, 1
  // that still gives three workgroups per CU
  int cus = 0, dev = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  p.group = 1;
  for (int g : {4, 2}) {
    if ((blocks + g - 1) / g * p.n_ftiles >= 3 * (int64_t)cus) {
      p.group = g;
      break;
    }
  }
  p.n_groups = (int32_t)((blocks + p.group - 1) / p.group);
  const int64_t groups8 = (p.n_groups + kXcds - 1) / kXcds * kXcds;
  const uint32_t gx = (uint32_t)(groups8 * p.n_ftiles);
  const size_t lds = (size_t)32 * fb * (p.K + 8) * 2;
  switch (fb) {
    case 6:
      hipLaunchKernelGGL((proj_kernel<6, MODE>), dim3(gx), dim3(64 * kWaves), lds, s, p);
      break;
    case 3:
      hipLaunchKernelGGL((proj_kernel<3, MODE>), dim3(gx), dim3(64 * kWaves), lds, s, p);
      break;
    case 2:
      hipLaunchKernelGGL((proj_kernel<2, MODE>), dim3(gx), dim3(64 * kWaves), lds, s, p);
      break;
    default:
      hipLaunchKernelGGL((proj_kernel<1, MODE>), dim3(gx), dim3(64 * kWaves), lds, s, p);
      break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_qkv_proj(const void *x, const void *w, const int32_t *order, void *q, void *k,
                           void *v, int64_t B, int64_t N, int64_t heads, int64_t d,
                           hipStream_t s) {
  ProjArgs p;
  p.in = static_cast<const __bf16 *>(x);
  p.order = order;
  p.w = static_cast<const __bf16 *>(w);
  p.out0 = static_cast<__bf16 *>(q);
  p.out1 = static_cast<__bf16 *>(k);
  p.out2 = static_cast<__bf16 *>(v);
  p.T = (int32_t)(B * N);
  p.N = (int32_t)N;
  p.C = (int32_t)(heads * d);
  p.K = p.C;
  p.F = 3 * p.C;
  p.heads = (int32_t)heads;
  p.d = (int32_t)d;
  return launch_fb<0>(p, s);
}

hipError_t launch_out_proj(const void *o, const void *w, const int32_t *order, void *y, int64_t B,
                           int64_t N, int64_t heads, int64_t d, int64_t c_out, hipStream_t s) {
  ProjArgs p;
  p.in = static_cast<const __bf16 *>(o);
  p.order = order;
  p.w = static_cast<const __bf16 *>(w);
  p.out0 = static_cast<__bf16 *>(y);
  p.out1 = p.out2 = nullptr;
  p.T = (int32_t)(B * N);
  p.N = (int32_t)N;
  p.C = (int32_t)(heads * d);
  p.K = p.C;
  p.F = (int32_t)c_out;
  p.heads = (int32_t)heads;
  p.d = (int32_t)d;
  return launch_fb<1>(p, s);
}

}  // namespace hla
