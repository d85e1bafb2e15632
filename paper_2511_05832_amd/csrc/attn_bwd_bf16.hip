// Block-sparse flash-attention backward, bf16 in / bf16 out, fp32 accumulation,
// on gfx950 bf16 matrix cores (v_mfma_f32_32x32x16_bf16).
//
// What it computes: the gradients of the forward pass (the paper times the
// backward of every attention it measures, Tables 1, 3, 6, 7, 9, 11) over the same
// tile structure - empty tiles skipped, full tiles unmasked, partial tiles with
// the element mask (Sec. 3.1; Eq. 1's per-block cost applies to both passes).
// With the forward's lse and delta_i = <dout_i, out_i> (sum_j P_ij dP_ij, since
// out_i = sum_j P_ij v_j):
//   P_ij  = exp(scale <q_i, k_j> - lse_i)   (0 where masked)
//   dS_ij = P_ij (<dout_i, v_j> - delta_i)
//   dq_i  = scale sum_j dS_ij k_j       dk_j = scale sum_i dS_ij q_i
//   dv_j  = sum_i P_ij dout_i
// Two kernels and no atomics, so every result is deterministic:
//   dq kernel    one workgroup per (b*h, query tile), walking that tile row's list
//                of key tiles (as the forward does); it also computes each row's
//                statistics (lse * log2 e, -delta) and stores them for the next;
//   dkdv kernel  one workgroup per (b*h, key tile), walking that key tile
//                column's list of query tiles (the transposed lists).
// P and dP are recomputed in both; the recomputation costs two of the seven
// products but removes every cross-workgroup reduction.
//
// Operand placement. In each kernel the operands that stay fixed over the walk
// (q and dout rows in dq; k and v rows in dkdv) live in registers as B operands,
// and the walked tiles are staged in LDS by global_load_lds_dwordx4 (no register
// round trip), in a ring kept ahead of the compute. A tile is read twice from
// LDS: by rows (A operand of S and dP) and transposed (A operand of the products
// that contract over the walked index, via ds_read_b64_tr_b16). One XOR swizzle
// of the 16-byte chunks serves both reads without bank conflicts:
//   d = 64: chunk ^= 2*(r%4) + (r/8)%2;   d = 32: chunk ^= 2*((r/2)%2) + (r/8)%2.
// The row reads touch rows {0..3, 8..11} (+16k) eight lanes at a time, which the
// low bit and (for d = 32) the row pairing make distinct; the transposing reads
// touch four consecutive rows times two adjacent chunks, which the upper two
// bits make distinct.
//
// Register-resident weights. The A rows of S (dq: key rows; dkdv: query rows) are
// fed permuted by row_perm, so the S and dP accumulators come out in the B-operand
// layout of the next product, and P / dS go to bf16 operands in place.
#include <algorithm>
#include <cstdlib>
#include <type_traits>

#include "attn_common.h"

namespace hla {
namespace {

constexpr int BN = 64;  // keys per key tile

template <int D>
__device__ __forceinline__ int swz(int r) {
  if (D == 64) return (2 * (r & 3)) | ((r >> 3) & 1);
  return (2 * ((r >> 1) & 1)) | ((r >> 3) & 1);
}

// A-operand byte offsets of a transposing read, relative to the first row of a
// 16-row step: lane i of 16-lane group g reads row 8(g/2) + i/4 (+4 for the
// second read), columns db*32 + 16(g%2) + 4(i%4). Row offsets that are multiples
// of 16 leave the swizzle unchanged, so a step adds a constant.
template <int D>
__device__ __forceinline__ int tr_base(int lane, int db) {
  const int g16 = lane >> 4, i16 = lane & 15;
  const int r = 8 * (g16 >> 1) + (i16 >> 2);
  const int cl = db * 32 + 16 * (g16 & 1) + 4 * (i16 & 3);
  return r * D * 2 + (((cl >> 3) ^ swz<D>(r)) * 16) + (cl & 7) * 2;
}

// Store a [d x 32] fp32 accumulator set (NDB blocks of 32x32, rows = d) scaled
// by `mul` as 32 bf16 rows of d, through this wave's LDS staging area `Os`
// (32 x (D + 8) bf16), to `dst` (row stride D). The caller barriers between
// the staging writes and the reads.
template <int D>
__device__ __forceinline__ void stage_rows(const f32x16 *acc, float mul, __bf16 *Os, int col,
                                           int half) {
  constexpr int OS = D + 8;
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 o4;
#pragma unroll
      for (int b = 0; b < 4; ++b) o4[b] = (__bf16)(acc[db][4 * g + b] * mul);
      *reinterpret_cast<bf16x4 *>(Os + col * OS + db * 32 + 8 * g + 4 * half) = o4;
    }
}
// Only the first `nrows` rows are written (rows past the end of the sequence in
// a ragged last tile are not). Row r goes to dst row r, or to dst row rows[r]
// when a row map is given (the fused reordering).
template <int D>
__device__ __forceinline__ void write_rows(const __bf16 *Os, __bf16 *dst, int lane, int nrows,
                                           const int32_t *rows = nullptr) {
  constexpr int OS = D + 8, CPR = D / 8;
  static_assert(32 * CPR % 64 == 0, "the rows' chunks split evenly over the lanes");
#pragma unroll
  for (int k = 0; k < 32 * CPR / 64; ++k) {
    const int i = lane + 64 * k;
    const int r = i / CPR, c = i % CPR;
    if (r < nrows) {
      const int64_t row = rows ? (int64_t)rows[r] : (int64_t)r;
      *reinterpret_cast<uint4 *>(dst + row * D + c * 8) =
          *reinterpret_cast<const uint4 *>(Os + r * OS + c * 8);
    }
  }
}

// ---------------------------------------------------------------------------
// dq: one workgroup per (b*h, query tile of BM = 32*NW rows); wave w owns 32
// queries. Per key tile, per wave:
//   S^T  = K Q^T      A = K rows (LDS), B = the wave's q (registers)
//   dP^T = V dout^T   A = V rows (LDS), B = the wave's dout (registers)
//   dS^T = P^T (dP^T - delta), P^T = exp2(S^T scale log2e - lse log2e)
//   dq^T += K^T dS^T  A = K^T (transposing LDS reads), B = dS^T (registers)
constexpr int kStagesDq = 3;

template <int D, int NW, bool GATHER>
__global__ void __launch_bounds__(64 * NW, NW == 4 ? 3 : 2) attn_bwd_dq_bf16(AttnBwdArgs a) {
  constexpr int BM = 32 * NW;
  constexpr int NT = 64 * NW;
  constexpr int CPR = D / 8;
  constexpr int TILE = BN * D * 2;
  constexpr int STAGE = 2 * TILE;  // K tile then V tile
  constexpr int CPW = BN * CPR / NT;
  constexpr int LPT = 2 * CPW;
  constexpr int NCH = D / 16;
  constexpr int NDB = D / 32;
  static_assert(BN * CPR % NT == 0, "tile copies must split evenly over the workgroup");
  static_assert((kStagesDq - 2) * LPT < 64, "too many copies in flight for vmcnt");
  // GATHER: the query tile's BM row indices, then four slots of BN indices for
  // key tiles (slot i % 4 holds tile list entry i).
  constexpr int IDXQ = kStagesDq * STAGE;
  constexpr int IDXK = IDXQ + BM * 4;
  constexpr int LDSB = GATHER ? IDXK + 4 * BN * 4 : kStagesDq * STAGE;

  __shared__ __attribute__((aligned(16))) char lds[LDSB];
  const int32_t *idx_q = reinterpret_cast<const int32_t *>(lds + IDXQ);
  auto idx_k = [&](int i) { return reinterpret_cast<const int32_t *>(lds + IDXK + (i & 3) * BN * 4); };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, half = lane >> 5;

  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = logical / a.n_qtiles;
  const int qt = logical - bh * a.n_qtiles;
  const int q0 = qt * BM;
  const int64_t slice = (int64_t)bh * a.N * D;
  const __bf16 *Q = static_cast<const __bf16 *>(a.q) + slice;
  const __bf16 *K = static_cast<const __bf16 *>(a.k) + slice;
  const __bf16 *V = static_cast<const __bf16 *>(a.v) + slice;
  const __bf16 *G = static_cast<const __bf16 *>(a.dout) + slice;

  const int qpos = q0 + wave * 32 + col;

  const PatternArgs &P = a.pat;
  const Region R = region_of<true>(P, qpos);

  const int nf = sload(a.n_full + qt), np = sload(a.n_part + qt), ntot = nf + np;
  const int32_t *frow = a.full_idx + (int64_t)qt * a.n_ktiles;
  const int32_t *prow = a.part_idx + (int64_t)qt * a.n_ktiles;
  auto tile_of = [&](int i) { return i < nf ? sload(frow + i) : sload(prow + i - nf); };

  // Row within the tile and chunk offset of this thread's copies. Rows past the
  // end of the sequence (ragged last key tile, always partial) read row N - 1
  // and are masked.
  int offr[CPW], offc[CPW];
#pragma unroll
  for (int j = 0; j < CPW; ++j) {
    const int p = (j * NW + wave) * 64 + lane;
    const int r = p / CPR, cs = p % CPR;
    offr[j] = r;
    offc[j] = (cs ^ swz<D>(r)) * 8;
  }
  // Copies of the K/V tile of list entry i (GATHER: row r of the tile is the
  // row its index slot names).
  auto issue_tile = [&](int i, int stage) {
    char *base = lds + stage * STAGE;
    int64_t roff[CPW];
    if constexpr (GATHER) {
      const int32_t *rows = idx_k(i);
#pragma unroll
      for (int j = 0; j < CPW; ++j) roff[j] = (int64_t)rows[offr[j]] * D + offc[j];
    } else {
      const int kt = tile_of(i);
#pragma unroll
      for (int j = 0; j < CPW; ++j) roff[j] = (int64_t)min(kt * BN + offr[j], a.N - 1) * D + offc[j];
    }
#pragma unroll
    for (int j = 0; j < CPW; ++j)
      lds_dma16(K + roff[j], lds_addr(base + (j * NW + wave) * 1024));
#pragma unroll
    for (int j = 0; j < CPW; ++j)
      lds_dma16(V + roff[j], lds_addr(base + TILE + (j * NW + wave) * 1024));
  };
  // GATHER: the row indices of list entry i (one per lane of the first wave)
  // into its slot; positions past the end of the sequence read entry N - 1.
  auto issue_idx = [&](int i) {
    if (wave == 0)
      lds_dma4(a.order + min(tile_of(i) * BN + lane, a.N - 1), lds_addr(lds + IDXK + (i & 3) * BN * 4));
  };

  int raddr[2][NCH];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int r = kb * 32 + row_perm(col);
#pragma unroll
    for (int c = 0; c < NCH; ++c) raddr[kb][c] = r * D * 2 + (((half * NCH + c) ^ swz<D>(r)) * 16);
  }
  int tbase[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) tbase[db] = tr_base<D>(lane, db);

  f32x16 acc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) acc[db] = f32x16{};
  const float sl2 = a.scale_log2;

  if constexpr (GATHER) {
    // Row indices of the query tile and of the first three key tiles, first.
    if (wave == 0) {
#pragma unroll
      for (int c = 0; c < BM / 64; ++c)
        lds_dma4(a.order + min(q0 + 64 * c + lane, a.N - 1), lds_addr(lds + IDXQ + 256 * c));
    }
#pragma unroll
    for (int i = 0; i < 3; ++i)
      if (i < ntot) issue_idx(i);
    wait_then_barrier<0>();
  }
#pragma unroll
  for (int p = 0; p < kStagesDq - 1; ++p)
    if (p < ntot) issue_tile(p, p);
  // The wave's own q and dout rows and row statistics, loaded after the first
  // copies so that both latencies overlap; one wait the compiler can see then
  // covers all of them, so it inserts no wait of its own inside the loop.
  // (a query row past the end of the sequence reads row N - 1 and stores nothing)
  const int64_t qrow = GATHER ? (int64_t)idx_q[wave * 32 + col] : (int64_t)min(qpos, a.N - 1);
  bf16x8 qop[NCH], gop[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    qop[c] = *reinterpret_cast<const bf16x8 *>(Q + qrow * D + half * (D / 2) + 8 * c);
    gop[c] = *reinterpret_cast<const bf16x8 *>(G + qrow * D + half * (D / 2) + 8 * c);
  }
  // This query's row statistics, computed here and stored for the dk/dv kernel:
  // delta = <dout, out> (this lane's half of d, then the other half's from lane
  // ^ 32) and lse * log2 e (+inf for a row with no allowed key, which makes every
  // recomputed weight exp2(s - inf) = 0 without a special case).
  const __bf16 *O = static_cast<const __bf16 *>(a.out) + slice;
  bf16x8 oop[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
    oop[c] = *reinterpret_cast<const bf16x8 *>(O + qrow * D + half * (D / 2) + 8 * c);
  const float lraw = a.lse[(int64_t)bh * a.N + qrow];
  wait_vmem_all();
  float dpart = 0.f;
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int e = 0; e < 8; ++e) dpart = __builtin_fmaf((float)oop[c][e], (float)gop[c][e], dpart);
  const float delta = dpart + __shfl_xor(dpart, 32);
  const float lse2 = lraw == -__builtin_inff() ? __builtin_inff() : lraw * 1.4426950408889634f;
  if (half == 0 && qpos < a.N)
    *reinterpret_cast<float2 *>(a.stats + 2 * ((int64_t)bh * a.N + qrow)) = make_float2(lse2, -delta);

  // One key tile. MASKED is a compile-time flag: full and partial tiles run
  // separate loop bodies (the lists hold the full tiles first), so neither
  // carries the other's registers (one body with a run-time mask branch copied
  // all 32 score accumulators on every full tile).
  auto step = [&](int it, auto masked) __attribute__((always_inline)) {
    const int stage = it % kStagesDq;
    wait_tiles_then_barrier<LPT, kStagesDq - 2>(min(ntot - 1 - it, kStagesDq - 2));
    // (GATHER: the indices of entry it + 2 arrived with the wait above - the
    // first wave issued them before entry it + 1's copies - those of it + 3 go
    // out first; slot (it + 3) % 4 last held entry it - 1's.)
    if constexpr (GATHER) {
      if (it + 3 < ntot) issue_idx(it + 3);
    }
    if (it + kStagesDq - 1 < ntot) issue_tile(it + kStagesDq - 1, (it + kStagesDq - 1) % kStagesDq);
    const char *st = lds + stage * STAGE;
    const int kt = tile_of(it);

    // the tile's two 32-key blocks one after the other (half the score
    // registers of both at once)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f32x16 s[1] = {f32x16{}}, dp = f32x16{};
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const bf16x8 kop = *reinterpret_cast<const bf16x8 *>(st + raddr[kb][c]);
        s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop, qop[c], s[0], 0, 0, 0);
        const bf16x8 vop = *reinterpret_cast<const bf16x8 *>(st + TILE + raddr[kb][c]);
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop, gop[c], dp, 0, 0, 0);
      }
      if constexpr (decltype(masked)::value) mask_blocks<1>(s, R, P, kt * BN + 32 * kb + 8 * half);
      bf16x8 dsop[2];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(s[0][v] * sl2 - lse2);
        dsop[v >> 3][v & 7] = (__bf16)(p * (dp[v] - delta));
      }
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const bf16x8 kto = lds_read_tr16x2(st + tbase[db] + (16 * (2 * kb + t)) * D * 2, D * 2);
          acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kto, dsop[t], acc[db], 0, 0, 0);
        }
    }
  };
  int it = 0;
  for (; it < nf; ++it) step(it, std::false_type{});
  for (; it < ntot; ++it) step(it, std::true_type{});

  wait_then_barrier<0>();
  __bf16 *Os = reinterpret_cast<__bf16 *>(lds) + wave * 32 * (D + 8);
  stage_rows<D>(acc, a.scale, Os, col, half);
  __syncthreads();
  if constexpr (GATHER)
    write_rows<D>(Os, static_cast<__bf16 *>(a.dq) + slice, lane, a.N - (q0 + wave * 32),
                  idx_q + wave * 32);
  else
    write_rows<D>(Os, static_cast<__bf16 *>(a.dq) + slice + (int64_t)(q0 + wave * 32) * D, lane,
                  a.N - (q0 + wave * 32));
}

// ---------------------------------------------------------------------------
// dkdv: one workgroup (4 waves) per (b*h, key tile of 64). Wave w owns the 32
// keys of block kb = w%2 and the query rows of half qh = w/2 of every query
// tile (BMQ/2 rows, QB blocks of 32). Per query tile, per wave and block:
//   S  = Q K^T       A = Q rows (LDS), B = the wave's k (registers)
//   dP = dout V^T    A = dout rows (LDS), B = the wave's v (registers)
//   P, dS as above, with lse and delta per query row from the staged stats
//   dv^T += dout^T P   A = dout^T (transposing reads), B = P (registers)
//   dk^T += Q^T dS     A = Q^T (transposing reads), B = dS (registers)
// The two query halves of a key block are summed through LDS at the end.
constexpr int kStagesKv = 2;

// Whether the dk/dv kernel's epilogue LDS (the query halves' exchange, then the
// rows' staging) fits one ring stage of a BMQ-row query tile.
template <int D, int BMQ>
constexpr bool dkdv_streams() {
  constexpr int stage = 2 * BMQ * D * 2 + BMQ * 8;
  constexpr int xch = 2 * 2 * (D / 32) * 16 * 64 * 4, rows = 4 * 32 * (D + 8) * 2;
  return (xch > rows ? xch : rows) <= stage;
}

template <int D, int BMQ, bool GATHER>
__global__ void __launch_bounds__(256, 2) attn_bwd_dkdv_bf16(AttnBwdArgs a) {
  constexpr int NT = 256;
  constexpr int CPR = D / 8;
  constexpr int QT = BMQ * D * 2;       // bytes of a Q (or dout) tile
  constexpr int SOFF = 2 * QT;          // stats after Q and dout: lse log2e of the rows,
  constexpr int SND = SOFF + BMQ * 4;   // then -delta of the rows
  constexpr int STAGE = 2 * QT + BMQ * 8;
  constexpr int CPW = BMQ * CPR / NT;   // 16-byte copies per thread per tile (Q or dout)
  constexpr int SL = BMQ / 2;           // stats values copied per wave (4 bytes each)
  constexpr int LPT = 2 * CPW + 1;
  constexpr int QB = BMQ / 64;
  constexpr int HALF = BMQ / 2;
  constexpr int NCH = D / 16;
  constexpr int NDB = D / 32;
  constexpr int XCH = 2 * 2 * NDB * 16 * 64 * 4;           // partial-sum exchange
  constexpr int EPI = XCH > 4 * 32 * (D + 8) * 2 ? XCH : 4 * 32 * (D + 8) * 2;
  constexpr int LDSR = kStagesKv * STAGE > EPI ? kStagesKv * STAGE : EPI;
  // GATHER: the key tile's BN row indices, then four slots of BMQ indices for
  // query tiles (slot i % 4 holds tile list entry i).
  constexpr int KIDX = LDSR;
  constexpr int QIDX = KIDX + BN * 4;
  constexpr int LDSB = GATHER ? QIDX + 4 * BMQ * 4 : LDSR;
  static_assert(CPW >= 1 && BMQ * CPR % NT == 0, "tile copies must split evenly");
  static_assert(SL <= 64, "stats copies exceed a wave");
  static_assert(4 * SL * 4 == BMQ * 8, "the waves' stats copies cover the tile's rows");
  // Several heads per workgroup when the epilogue's LDS fits one ring stage (it
  // then uses the stage the item's last tile left while the other one receives
  // the next item's first tile).
  constexpr bool STREAMS = dkdv_streams<D, BMQ>();
  static_assert(!STREAMS || EPI <= STAGE, "the epilogue must fit one stage");

  __shared__ __attribute__((aligned(16))) char lds[LDSB];
  const int32_t *idx_k = reinterpret_cast<const int32_t *>(lds + KIDX);
  auto idx_q = [&](int i) { return reinterpret_cast<const int32_t *>(lds + QIDX + (i & 3) * BMQ * 4); };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, half = lane >> 5;
  const int kb = wave & 1, qh = wave >> 1;

  // The workgroup runs its key tile for a group of consecutive heads (the
  // items; one without STREAMS), the key tile fastest in the grid as in the
  // other kernels. (GATHER: every head has the same rows and lists.)
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int grp = logical / a.n_ktiles;
  const int kt = logical - grp * a.n_ktiles;
  int bh = grp, nitems = 1;
  if constexpr (STREAMS) {
    // groups of q + 1 heads first, then of q (q = BH / hgroups, r = BH % hgroups)
    const int q = a.BH / a.hgroups, r = a.BH - q * a.hgroups;
    bh = grp * q + min(grp, r);
    nitems = q + (grp < r ? 1 : 0);
  }
  const int k0 = kt * BN;
  const int64_t ND = (int64_t)a.N * D;  // elements per head
  const int64_t slice = (int64_t)bh * ND;
  const __bf16 *Q = static_cast<const __bf16 *>(a.q) + slice;
  const __bf16 *K = static_cast<const __bf16 *>(a.k) + slice;
  const __bf16 *V = static_cast<const __bf16 *>(a.v) + slice;
  const __bf16 *G = static_cast<const __bf16 *>(a.dout) + slice;
  const float *S = a.stats + 2 * (int64_t)bh * a.N;

  const int kpos = k0 + kb * 32 + col;

  const PatternArgs &P = a.pat;
  const Region R = region_of<false>(P, kpos);

  const int nf = sload(a.n_full_t + kt), np = sload(a.n_part_t + kt), ntot = nf + np;
  const int32_t *fcol = a.full_idx_t + (int64_t)kt * a.n_qtiles;
  const int32_t *pcol = a.part_idx_t + (int64_t)kt * a.n_qtiles;
  auto tile_of = [&](int i) { return i < nf ? sload(fcol + i) : sload(pcol + i - nf); };

  // Query rows past the end of the sequence (ragged last query tile, always
  // partial) read row N - 1 and are masked.
  int offr[CPW], offc[CPW];
#pragma unroll
  for (int j = 0; j < CPW; ++j) {
    const int p = (j * 4 + wave) * 64 + lane;
    const int r = p / CPR, cs = p % CPR;
    offr[j] = r;
    offc[j] = (cs ^ swz<D>(r)) * 8;
  }
  // Copies of the query tile of list entry i of item h: Q, dout and the rows'
  // stats (GATHER: row r of the tile is the row index slot `slot` names).
  auto issue_tile = [&](int i, int stage, int h, int slot) {
    char *base = lds + stage * STAGE;
    const int qt = tile_of(i);
    const __bf16 *Qh = Q + h * ND, *Gh = G + h * ND;
    const float *Sh = S + 2 * (int64_t)h * a.N;
    int64_t roff[CPW];
    if constexpr (GATHER) {
      const int32_t *rows = idx_q(slot);
#pragma unroll
      for (int j = 0; j < CPW; ++j) roff[j] = (int64_t)rows[offr[j]] * D + offc[j];
    } else {
#pragma unroll
      for (int j = 0; j < CPW; ++j) roff[j] = (int64_t)min(qt * BMQ + offr[j], a.N - 1) * D + offc[j];
    }
#pragma unroll
    for (int j = 0; j < CPW; ++j)
      lds_dma16(Qh + roff[j], lds_addr(base + (j * 4 + wave) * 1024));
#pragma unroll
    for (int j = 0; j < CPW; ++j)
      lds_dma16(Gh + roff[j], lds_addr(base + QT + (j * 4 + wave) * 1024));
    // stats value f of the tile = component f / BMQ of row f % BMQ, so that the
    // stage holds lse log2e of every row, then -delta of every row
    if (lane < SL) {
      const int f = wave * SL + lane, r = f % BMQ;
      const int64_t row = GATHER ? (int64_t)idx_q(slot)[r] : (int64_t)min(qt * BMQ + r, a.N - 1);
      lds_dma4(Sh + 2 * row + f / BMQ, lds_addr(base + SOFF + wave * SL * 4));
    }
  };
  // GATHER: the row indices of list entry i (first wave, one per lane) into
  // index slot `slot`; positions past the end of the sequence read entry N - 1.
  auto issue_idx = [&](int i, int slot) {
    if (wave == 0) {
#pragma unroll
      for (int c = 0; c < BMQ / 64; ++c)
        lds_dma4(a.order + min(tile_of(i) * BMQ + 64 * c + lane, a.N - 1),
                 lds_addr(lds + QIDX + (slot & 3) * BMQ * 4 + 256 * c));
    }
  };
  // Element k of the stream after entry it of item h (the items' lists one after
  // the other): its item hh and entry ii; false past the last item (and for an
  // empty list).
  auto elem = [&](int h, int it, int k, int &hh, int &ii) {
    hh = h;
    ii = it + k;
    if (ntot <= 0) return false;
    while (ii >= ntot) {
      ii -= ntot;
      ++hh;
    }
    return hh < nitems;
  };

  int raddr[QB][NCH];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int r = qh * HALF + qb * 32 + row_perm(col);
#pragma unroll
    for (int c = 0; c < NCH; ++c) raddr[qb][c] = r * D * 2 + (((half * NCH + c) ^ swz<D>(r)) * 16);
  }
  int tbase[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) tbase[db] = tr_base<D>(lane, db) + qh * HALF * D * 2;

  f32x16 dk[NDB], dv[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) {
    dk[db] = f32x16{};
    dv[db] = f32x16{};
  }
  const float sl2 = a.scale_log2;

  // (GATHER: the element counter e of the stream picks the index slot, e % 4)
  if constexpr (GATHER) {
    // Row indices of the key tile and of the stream's first two query tiles,
    // first.
    if (wave == 0)
      lds_dma4(a.order + min(k0 + lane, a.N - 1), lds_addr(lds + KIDX));
    if (ntot > 0) {
      int hh, ii;
      for (int k = 0; k < 2; ++k)
        if (elem(0, 0, k, hh, ii)) issue_idx(ii, k);
    }
    wait_then_barrier<0>();
  }
  if (ntot > 0) issue_tile(0, 0, 0, 0);
  // The wave's own k and v rows of item h (the first item's loaded after the
  // first copy so that both latencies overlap; one wait the compiler can see
  // then covers both, so it inserts no wait of its own inside the loop).
  // (a key row past the end of the sequence reads row N - 1 and stores nothing)
  const int64_t krow = GATHER ? (int64_t)idx_k[kb * 32 + col] : (int64_t)min(kpos, a.N - 1);
  bf16x8 kop[NCH], vop[NCH];
  // (byte offset within a head: below 2^31, as N * d <= 2^30)
  const uint32_t kvoff = (uint32_t)(krow * D + half * (D / 2)) * 2u;
  auto load_kv = [&](int h) {
    const char *Kh = reinterpret_cast<const char *>(K + h * ND) + kvoff;
    const char *Vh = reinterpret_cast<const char *>(V + h * ND) + kvoff;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      kop[c] = *reinterpret_cast<const bf16x8 *>(Kh + 16 * c);
      vop[c] = *reinterpret_cast<const bf16x8 *>(Vh + 16 * c);
    }
  };
  load_kv(0);
  wait_vmem_all();

  // One query tile, list entry it of item h; full and partial tiles run
  // separate loop bodies (as in the dq kernel). The items' tiles are one
  // stream through the two-stage ring: each step copies the next tile (the
  // item's next entry, or the next item's entry 0) into the other stage.
  int h = 0, cur = 0, e = 0;  // item, stage of the tile read next, its element
  auto step = [&](int it, auto masked) __attribute__((always_inline)) {
    const int stage = cur;
    cur ^= 1;
    wait_then_barrier<0>();
    // (GATHER: element e + 1's indices arrived with the wait above; element
    // e + 2's go out first, into slot (e + 2) % 4, last read for element e - 2.)
    int hh, ii;
    if constexpr (GATHER) {
      if (elem(h, it, 2, hh, ii)) issue_idx(ii, e + 2);
    }
    if (elem(h, it, 1, hh, ii)) issue_tile(ii, cur, hh, e + 1);
    ++e;
    const char *st = lds + stage * STAGE;
    const int qt = tile_of(it);

    // dP - delta directly: each dP accumulator starts at -delta of its rows. Slot
    // v of block qb is row qh*HALF + 32qb + 16(v/8) + 8half + v%8 (two runs of
    // eight rows), i.e. two 16-byte reads per run from the staged -delta.
    f32x16 s[QB], dp[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      s[qb] = f32x16{};
      const float4 *nd = reinterpret_cast<const float4 *>(st + SND + (qh * HALF + 32 * qb + 8 * half) * 4);
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const float4 lo = nd[4 * g], hi = nd[4 * g + 1];
        dp[qb][8 * g + 0] = lo.x; dp[qb][8 * g + 1] = lo.y; dp[qb][8 * g + 2] = lo.z; dp[qb][8 * g + 3] = lo.w;
        dp[qb][8 * g + 4] = hi.x; dp[qb][8 * g + 5] = hi.y; dp[qb][8 * g + 6] = hi.z; dp[qb][8 * g + 7] = hi.w;
      }
    }
#pragma unroll
    for (int c = 0; c < NCH; ++c)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const bf16x8 qa = *reinterpret_cast<const bf16x8 *>(st + raddr[qb][c]);
        s[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, kop[c], s[qb], 0, 0, 0);
        const bf16x8 ga = *reinterpret_cast<const bf16x8 *>(st + QT + raddr[qb][c]);
        dp[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ga, vop[c], dp[qb], 0, 0, 0);
      }
    if constexpr (decltype(masked)::value) mask_blocks<QB>(s, R, P, qt * BMQ + qh * HALF + 8 * half);

    bf16x8 pop[2 * QB], dsop[2 * QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        // rows qh*HALF + 32qb + 16g + 8half + (0..7): two 16-byte reads of their
        // lse log2e, every lane of a half on the same address
        const float4 *ls = reinterpret_cast<const float4 *>(
            st + SOFF + (qh * HALF + 32 * qb + 16 * g + 8 * half) * 4);
        const float4 la = ls[0], lb = ls[1];
        const float l2[8] = {la.x, la.y, la.z, la.w, lb.x, lb.y, lb.z, lb.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int v = 8 * g + e;
          const float p = __builtin_amdgcn_exp2f(s[qb][v] * sl2 - l2[e]);
          pop[2 * qb + g][e] = (__bf16)p;
          dsop[2 * qb + g][e] = (__bf16)(p * dp[qb][v]);
        }
      }

#pragma unroll
    for (int t = 0; t < 2 * QB; ++t)
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const bf16x8 gt = lds_read_tr16x2(st + QT + tbase[db] + (16 * t) * D * 2, D * 2);
        dv[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(gt, pop[t], dv[db], 0, 0, 0);
        const bf16x8 qto = lds_read_tr16x2(st + tbase[db] + (16 * t) * D * 2, D * 2);
        dk[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qto, dsop[t], dk[db], 0, 0, 0);
      }
  };
  for (h = 0; h < nitems; ++h) {
    // (a wait the compiler sees, at every item: it covers the k and v rows
    // loaded during the previous item's epilogue - and that item's first tile
    // and stores - so the compiler adds no wait of its own in the tile loop)
    wait_vmem_all();
    int it = 0;
    for (; it < nf; ++it) step(it, std::false_type{});
    for (; it < ntot; ++it) step(it, std::true_type{});
    // the next item's k and v rows, in flight during this item's epilogue (the
    // products no longer read this item's)
    if (h + 1 < nitems) load_kv(h + 1);

    // Sum the two query halves: half 1 hands its dk to half 0, half 0 hands its
    // dv to half 1; then half 0 writes dk and half 1 writes dv. Through the
    // stage the item's last tile used (the other one may be receiving the next
    // item's first tile), with barriers that wait for LDS only.
    char *ep = STREAMS && nitems > 1 ? lds + (cur ^ 1) * STAGE : lds;
    // (the lane index passed through an empty asm: the epilogue's addresses are
    // then computed here, per item, instead of being kept in registers across
    // the loop, where they would be spilled and their reloads would wait for
    // the copies in flight)
    int ln = lane;
    asm volatile("" : "+v"(ln));
    const int lcol = ln & 31, lhalf = ln >> 5;
    wait_then_barrier<63>();
    float *xch = reinterpret_cast<float *>(ep);
    auto xidx = [&](int which, int db, int v) {
      return (((kb * 2 + which) * NDB + db) * 16 + v) * 64 + ln;
    };
    // (qh is wave-uniform: one branch around whole loops, not one per element)
    const int give = qh == 1 ? 0 : 1, keep = 1 - give;
    if (qh == 1) {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) xch[xidx(give, db, v)] = dk[db][v];
    } else {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) xch[xidx(give, db, v)] = dv[db][v];
    }
    wait_then_barrier<63>();
    f32x16 res[NDB];
    if (qh == 0) {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) res[db][v] = dk[db][v] + xch[xidx(keep, db, v)];
    } else {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) res[db][v] = dv[db][v] + xch[xidx(keep, db, v)];
    }
    wait_then_barrier<63>();
    __bf16 *Os = reinterpret_cast<__bf16 *>(ep) + wave * 32 * (D + 8);
    stage_rows<D>(res, qh == 0 ? a.scale : 1.f, Os, lcol, lhalf);
    wait_then_barrier<63>();
    __bf16 *dst = static_cast<__bf16 *>(qh == 0 ? a.dk : a.dv) + slice + h * ND;
    if constexpr (GATHER)
      write_rows<D>(Os, dst, ln, a.N - (k0 + kb * 32), idx_k + kb * 32);
    else
      write_rows<D>(Os, dst + (int64_t)(k0 + kb * 32) * D, ln, a.N - (k0 + kb * 32));
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      dk[db] = f32x16{};
      dv[db] = f32x16{};
    }
  }
}

template <int D, int NW>
hipError_t launch_dq(const AttnBwdArgs &a, hipStream_t s) {
  const int64_t blocks = (int64_t)a.BH * a.n_qtiles;
  if (a.order)
    hipLaunchKernelGGL((attn_bwd_dq_bf16<D, NW, true>), dim3((uint32_t)blocks), dim3(64 * NW), 0, s, a);
  else
    hipLaunchKernelGGL((attn_bwd_dq_bf16<D, NW, false>), dim3((uint32_t)blocks), dim3(64 * NW), 0, s, a);
  return hipGetLastError();
}

// Heads per dk/dv workgroup (the 1-D patterns; the others keep one). A
// workgroup's set-up - its k and v rows and the first query tile's latency - is
// paid once for all its heads, while too few workgroups leave resident slots
// empty. With `slots` = CUs x resident workgroups per CU: the smallest count
// dividing B*heads that puts every workgroup in one round, within
// kHeadsWorkBwd query tiles of work per workgroup (a key's query span from the
// pattern) and 8 heads; else the largest dividing count within that cap.
// HLA_ATTN_BWD_HEADS_PER_WORKGROUP (1 .. 64) overrides it.
constexpr int kHeadsWorkBwd = 72;
int dkdv_heads_per_workgroup(const AttnBwdArgs &a, int BMQ, int per_cu) {
  if (const char *env = std::getenv("HLA_ATTN_BWD_HEADS_PER_WORKGROUP")) {
    const int h = std::atoi(env);
    if (h >= 1 && h <= 64) return h;
  }
  if (!pattern_is_1d(a.pat.kind)) return 1;
  const int64_t span = a.pat.kind == HLA_HILBERT_SLIDE ? 2 * (int64_t)a.pat.p0 + 1 : (int64_t)a.pat.p0;
  const int64_t tiles = (std::min<int64_t>(span, a.N) + BN + BMQ - 1) / BMQ;
  const int cap = (int)std::max<int64_t>(1, std::min<int64_t>(std::min<int64_t>(8, kHeadsWorkBwd / tiles), a.BH));
  const int64_t slots = (int64_t)device_cu_count() * std::max(per_cu, 1);
  const int64_t items = (int64_t)a.BH * a.n_ktiles;
  if (items <= slots) return 1;
  for (int d = 1; d <= cap; ++d)
    if (a.BH % d == 0 && (int64_t)(a.BH / d) * a.n_ktiles <= slots) return d;
  for (int d = cap; d > 1; --d)
    if (a.BH % d == 0) return d;
  return 1;
}

template <int D, int BMQ>
hipError_t launch_dkdv(const AttnBwdArgs &a_in, hipStream_t s) {
  AttnBwdArgs a = a_in;
  a.hgroups = a.BH;
  if (dkdv_streams<D, BMQ>()) {
    // resident workgroups per CU for each kernel, read once per instantiation
    static int per_cu[2] = {0, 0};
    const int g = a.order ? 1 : 0;
    if (!per_cu[g]) {
      int n = 0;
      const void *f = a.order ? reinterpret_cast<const void *>(&attn_bwd_dkdv_bf16<D, BMQ, true>)
                              : reinterpret_cast<const void *>(&attn_bwd_dkdv_bf16<D, BMQ, false>);
      per_cu[g] = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, f, 256, 0) == hipSuccess && n > 0 ? n : 1;
    }
    const int h = dkdv_heads_per_workgroup(a, BMQ, per_cu[g]);
    a.hgroups = (a.BH + h - 1) / h;  // groups of ceil or floor of BH / hgroups heads
  }
  const int64_t blocks = (int64_t)a.hgroups * a.n_ktiles;
  if (a.order)
    hipLaunchKernelGGL((attn_bwd_dkdv_bf16<D, BMQ, true>), dim3((uint32_t)blocks), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((attn_bwd_dkdv_bf16<D, BMQ, false>), dim3((uint32_t)blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int D, int BM>
hipError_t launch_all(const AttnBwdArgs &a, hipStream_t s) {
  // the dq kernel also writes the row statistics the dk/dv kernel reads
  hipError_t e = launch_dq<D, BM / 32>(a, s);
  if (e != hipSuccess) return e;
  return launch_dkdv<D, BM>(a, s);
}

}  // namespace

hipError_t launch_attn_bwd_bf16(const AttnBwdArgs &a, int d, int tile_m, int tile_n,
                                hipStream_t s) {
  if (tile_n != BN) return hipErrorInvalidValue;
  if (d == 64 && tile_m == 128) return launch_all<64, 128>(a, s);
  if (d == 64 && tile_m == 64) return launch_all<64, 64>(a, s);
  if (d == 32 && tile_m == 128) return launch_all<32, 128>(a, s);
  if (d == 32 && tile_m == 64) return launch_all<32, 64>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace hla
