// Block-sparse flash-attention forward, bf16 in / bf16 out, fp32 accumulation,
// on gfx950 bf16 matrix cores (v_mfma_f32_32x32x16_bf16).
//
// What it computes (Sec. 3.1; Eq. 1): for every (b, h) and query tile, walk the
// non-empty key tiles of that tile row only - the full ones without a mask,
// then the partial ones with the element mask - and keep a running (online)
// softmax, so empty tiles cost neither loads nor arithmetic.
//
// Work decomposition. One workgroup = one query tile of BM = 32*NW rows of one
// (b, h); wave w owns 32 query rows. Key tiles are BN = 64 keys.
//
// Per key tile, per wave:
//   S^T = K Q^T    (keys x queries): 2 key blocks of 32 x D/16 MFMAs. A = K rows
//                  from LDS, B = the wave's Q (kept in registers all kernel,
//                  after one pass through LDS at the start).
//   softmax        lane l owns query l%32; its 32 scores of the tile sit in its
//                  own accumulators (16 per key block, the other half of the keys
//                  in lane l^32), so row max / sum need one cross-half exchange.
//   O^T += V^T P^T (d x queries): D/32 blocks x 4 MFMAs. A = V^T read from LDS
//                  with the transposing ds_read_b64_tr_b16, B = P straight from
//                  the S^T accumulators (see below).
//
// Register-resident P. The accumulator of a 32x32 MFMA holds, in lane
// (col = l%32, half = l/32) and slot v, row 8*(v/4) + 4*half + v%4. The K rows
// fed to S^T are permuted (row_perm) so that accumulator slot v of lane half
// `half` is key 16*(v/8) + 8*half + v%8 of the block: eight consecutive keys per
// run, which is exactly the B-operand layout of the PV MFMA over 16 keys. So P
// goes from fp32 accumulators to bf16 operands in place, with no LDS trip.
// The contraction over d in S^T is likewise permuted (lane half `half` holds d
// in [half*D/2, (half+1)*D/2)), so each lane loads its Q slice as one
// contiguous run.
//
// K/V staging. K and V tiles go from global memory straight into LDS with
// global_load_lds_dwordx4 (no register round trip), into a ring of kStages
// stages kept kStages-1 tiles ahead. The Q tile takes the same path once, into
// the stage the third key tile fills later. The copies are issued from inline
// assembly: the compiler's wait insertion would otherwise treat each
// transposing V read as possibly overlapping a copy in flight and wait for all
// of them - including the tile prefetched two steps ahead - on every tile. Both are stored row-major, 16-byte chunks
// XOR-swizzled per row so that the K operand reads (ds_read_b128, eight lanes on
// eight rows) and the transposing V reads (ds_read_b64_tr_b16, sixteen lanes on
// four rows) each touch distinct bank groups; the swizzle is applied on the
// source side (each lane fetches the chunk that belongs in its LDS slot). Before
// each tile, a wave waits only for its own loads of that tile (an explicit
// vmcnt that leaves the later tiles in flight), then one barrier makes the
// stage visible to all waves.
//
// Tile-list entries are read with scalar loads. Accumulators live in ordinary
// VGPRs (the library is built with the VGPR form of MFMA). Full tiles and
// partial tiles run separate loop bodies (the lists hold the full tiles first),
// so the unmasked body carries no mask code.
//
// Epilogue. O is normalised and stored straight from the accumulators: one
// exchange between the two lane halves gives each lane 16 contiguous bytes of
// its query's row.
//
// Masking (partial tiles only). For the 1-D Hilbert patterns each query's
// allowed keys are one interval [lo, hi] computed once per lane; for the
// row-major patterns they are one rectangle of grid cells. Masked scores are
// -inf before the row max; a query with no allowed key so far keeps m = -inf and
// contributes exactly zero.
//
// Ragged tilings (N not a multiple of the tile): a key tile reaching past the
// end of the sequence is always in the partial list, its rows past N - 1 are
// copied from row N - 1 and the mask (every allowed region is clipped at N - 1)
// drops them; query rows past N - 1 load row N - 1 and store nothing. Every
// global access stays inside the tensors.
//
// Grid: one workgroup per (b*h, query tile), remapped so each XCD (workgroups
// are dealt round-robin to the 8 XCDs) receives a contiguous range of query
// tiles: neighbouring tiles share key/value tiles (a window is two query tiles;
// a band overlaps its neighbour almost entirely), and the reuse stays in one
// XCD's L2.
#include <algorithm>
#include <cstdlib>
#include <type_traits>

#include "attn_common.h"
#include "hilbert_common.h"
#include "tiles_common.h"

namespace hla {
namespace {


constexpr int BN = 64;
constexpr float kRescaleSlack = 8.f;  // log2 units the softmax reference may lag the max
// Largest running weight sum per lane (its l, after adding the tile) the
// max-free softmax step accepts against a stale reference (2^32: far from fp32
// overflow in O and l).
constexpr float kFastBound = 4294967296.f;
// LDS ring depth. Three 16 KiB stages (d = 64) let three workgroups share a
// CU's 160 KiB; with the launch bound below that is the occupancy that measured
// fastest. Four stages at two workgroups per CU were slower, also with a
// software-pipelined body that computes the next tile's scores on the matrix
// cores during the current tile's softmax; so were two stages at four per CU.
constexpr int kStages = 3;

// Combine a value of lane l with lane l ^ 32 (the other half of a query's keys).
__device__ __forceinline__ float xhalf_max(float x) { return fmaxf(x, __shfl_xor(x, 32)); }
__device__ __forceinline__ float xhalf_sum(float x) { return x + __shfl_xor(x, 32); }

// RPB: table entries a staged bias window may hold (per buffer).
constexpr int kWinCap = 1024;

// HIL: list entries whose curve blocks are tabulated in LDS by the prologue
// (later entries, in rows with longer lists, walk the curve per tile).
constexpr int kBlkTab = 256;

// Bounding box {r_min, r_max, c_min, c_max} of the 64 lanes' grid cells (r, c <
// 2^15), in every lane: both coordinates' min and max at once, as packed 16-bit
// pairs. All 64 lanes must be active.
__device__ __forceinline__ int4 wave_box(int32_t r, int32_t c) {
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  u16x2 lo = {(unsigned short)r, (unsigned short)c}, hi = lo;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const u16x2 l2 = __builtin_bit_cast(u16x2, __shfl_xor(__builtin_bit_cast(int, lo), o));
    const u16x2 h2 = __builtin_bit_cast(u16x2, __shfl_xor(__builtin_bit_cast(int, hi), o));
    lo = __builtin_elementwise_min(lo, l2);
    hi = __builtin_elementwise_max(hi, h2);
  }
  return int4{lo.x, hi.x, lo.y, hi.y};
}

// Per-row XOR swizzle of the 16-byte chunks of a K / V tile row in LDS.
template <int D>
__device__ __forceinline__ int swz_k(int r) {
  if (D == 64) return (r & 3) | (((r >> 3) & 1) << 2);
  return ((r >> 1) & 1) | (((r >> 3) & 1) << 1);
}
template <int D>
__device__ __forceinline__ int swz_v(int r) {
  if (D == 64) return 2 * (r & 3);
  return 2 * ((r >> 1) & 1);
}

// Per-row XOR swizzle of the 16-byte chunks of the Q tile in LDS: the operand
// reads take eight consecutive rows at a time (one chunk each), which this
// spreads over distinct bank groups.
template <int D>
__device__ __forceinline__ int swz_q(int r) {
  if (D == 64) return r & 7;
  return (r >> 1) & 3;
}

// Launch bound (second argument: minimum waves per SIMD): three waves, i.e. at
// most 168 VGPRs per lane and three 4-wave workgroups per CU.
//
// MODE ATTN_GATHER: the tensors are stored in grid (row-major) order and
// sequence position i lives in row a.order[i] (the reordering fused into the
// loads and stores). Each key tile's 64 row indices are copied into LDS one step
// ahead of its K/V copies (by the first wave; issued before that step's K/V
// copies, so the same vmcnt counts cover them), and the Q tile's indices in the
// prologue, which also give each lane the row its output goes to.
//
// MODE ATTN_RPB: tensors in sequence order, and every score gets the global
// relative position bias table[h][r_i - r_j + H - 1][c_i - c_j + W - 1] of the
// grid cells (r, c) of order[i], order[j]. With off(g) = g + (W - 1) * (g / W)
// for a grid id g, that entry is table[h][C + off(q) - off(k)], C = (H - 1)(2W - 1)
// + W - 1. Each wave copies a quarter of a key tile's grid ids into LDS with the
// tile's K/V copies; each lane reads its 32 keys' ids from there and loads the
// 32 bias values (ordinary loads: the compiler waits for them - and, the vmcnt
// counter being in order, for the copies issued before them - before the
// softmax, so this mode issues each tile's copies at the end of the step two
// tiles earlier rather than at its start).
template <int D, int NW, int MODE>
// (waves per SIMD the launch bound asks for: what the registers and LDS allow -
// the RPB mode's windows leave room for two workgroups per CU)
__global__ void __launch_bounds__(64 * NW, MODE == ATTN_RPB ? (NW == 4 ? 2 : 1) : (NW == 4 ? 3 : 2))
    attn_fwd_bf16(AttnArgs a) {
  constexpr bool HIL = MODE == ATTN_HILBERT;
  // one query tile for several heads per workgroup (see the end of the kernel)
  constexpr bool STREAM = HIL;
  constexpr bool GATHER = MODE == ATTN_GATHER;
  constexpr bool RPB = MODE == ATTN_RPB;
  constexpr bool IDX = GATHER || RPB;
  constexpr int BM = 32 * NW;
  constexpr int NT = 64 * NW;
  constexpr int CPR = D / 8;                  // 16-byte chunks per K/V row
  constexpr int TILE = BN * D * 2;            // bytes of one K or V tile
  constexpr int STAGE = 2 * TILE;             // K tile then V tile
  constexpr int CPW = BN * CPR / NT;          // 16-byte copies per thread per tile (K or V)
  constexpr int LPT = 2 * CPW;                // vector memory ops per wave per tile
  constexpr int LQ = BM * CPR / NT;           // 16-byte copies per thread of the Q tile
  constexpr int NCH = D / 16;                 // MFMA steps over d for S^T
  constexpr int NDB = D / 32;                 // d blocks of O^T
  static_assert(BN * CPR % NT == 0 && BM * CPR % NT == 0, "copies must split evenly");
  static_assert(BM * D * 2 <= STAGE, "the Q tile must fit one stage");
  static_assert(kStages == 3, "the loop keeps exactly one tile in flight behind the current");
  static_assert(LPT < 64, "too many copies in flight for vmcnt");
  // Row-index area (GATHER): the Q tile's BM indices, then four slots of BN
  // indices for key tiles (slot i % 4 holds tile list entry i).
  constexpr int IDXQ = kStages * STAGE;
  constexpr int IDXK = IDXQ + BM * 4;
  // RPB: parameters {dr0, dc0, wc, n} of four tiles' bias windows, each key's
  // window term for them (four slots of BN), the waves' query boxes, and two
  // window buffers of kWinCap table entries.
  constexpr int WINP = IDXK + 4 * BN * 4;
  constexpr int WINB = WINP + 4 * 16;
  constexpr int QBOX = WINB + 4 * BN * 4;
  constexpr int WIN = QBOX + NW * 16;
  // HIL: the curve blocks of the first kBlkTab list entries, after the ring: the
  // grid row of the block's origin cell (a multiple of 8) ORed with the state
  // entering the block; then the row's runs (nf, ntot, t_lo, f_lo, f_hi).
  constexpr int BLKT = kStages * STAGE;
  constexpr int LDSB = RPB   ? WIN + 2 * kWinCap * 4
                       : IDX ? IDXK + 4 * BN * 4
                       : HIL ? BLKT + kBlkTab * 4 + 32
                             : kStages * STAGE;
  static_assert(!HIL || BN == 64, "a key tile must be one 8 x 8 block of the curve");

  __shared__ __attribute__((aligned(16))) char lds[LDSB];
  const int32_t *idx_q = reinterpret_cast<const int32_t *>(lds + IDXQ);
  auto idx_k = [&](int i) { return reinterpret_cast<const int32_t *>(lds + IDXK + (i & 3) * BN * 4); };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, half = lane >> 5;

  // (STREAM: a workgroup runs its query tile for one of a.hgroups near-equal
  // groups of consecutive heads, the items, starting at head bh. The query
  // tile varies fastest, as in the other modes, so each XCD's contiguous share
  // of the grid reads the keys of few heads.)
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int grp = logical / a.n_qtiles;
  const int qt = logical - grp * a.n_qtiles;
  int bh = grp, nitems = 1;
  if constexpr (STREAM) {
    bh = (int)((int64_t)grp * a.BH / a.hgroups);
    nitems = (int)((int64_t)(grp + 1) * a.BH / a.hgroups) - bh;
  }
  const int64_t slice = (int64_t)bh * a.N * D;
  const __bf16 *Q = static_cast<const __bf16 *>(a.q) + slice;
  const __bf16 *K = static_cast<const __bf16 *>(a.k) + slice;
  const __bf16 *V = static_cast<const __bf16 *>(a.v) + slice;

  // This lane's query. Its Q operand (d = half*D/2 + 8c + s for step c) is
  // staged through LDS below.
  const int qpos = qt * BM + wave * 32 + col;

  // Allowed-key region of this query (used on partial tiles only).
  const PatternArgs &P = a.pat;
  const Region R = region_of<true>(P, qpos);

  // Tile lists, read through the scalar unit: the full tiles, then the partial.
  // (HIL: set by the prologue.)
  int nf = 0, ntot = 0, t_lo = 0, f_lo = 0, f_hi = -1;
  if constexpr (!HIL) {
    nf = sload(a.n_full + qt);
    ntot = nf + sload(a.n_part + qt);
  }
  const int32_t *frow = HIL ? nullptr : a.full_idx + (int64_t)qt * a.n_ktiles;
  const int32_t *prow = HIL ? nullptr : a.part_idx + (int64_t)qt * a.n_ktiles;
  auto tile_of = [&](int i) {
    if constexpr (HIL) {
      if (i < nf) return f_lo + i;
      const int j = i - nf, before = f_lo - t_lo;
      return j < before ? t_lo + j : f_hi + 1 + (j - before);
    } else {
      return i < nf ? sload(frow + i) : sload(prow + i - nf);
    }
  };

  // Per-thread source offsets (elements, within a tile) of this thread's K and V
  // chunk copies: LDS slot p = (j*NW + wave)*64 + lane holds row p / CPR, chunk
  // (p % CPR) ^ swizzle(row).
  // (GATHER: row r of a tile is the row named by its index slot instead.)
  int krow[CPW], kch[CPW], vch[CPW];
#pragma unroll
  for (int j = 0; j < CPW; ++j) {
    const int p = (j * NW + wave) * 64 + lane;
    const int r = p / CPR, cs = p % CPR;
    krow[j] = r;
    kch[j] = (cs ^ swz_k<D>(r)) * 8;
    vch[j] = (cs ^ swz_v<D>(r)) * 8;
  }
  // Copies of the K/V tile of list entry i into a ring stage, each from the
  // wave-uniform slice base plus this lane's 32-bit byte offset (a slice holds at
  // most 2^30 elements).
  // (Plain mode: a tile inside the sequence takes its first row into the scalar
  // base, so its offsets are the loop-invariant in-tile ones; the ragged last
  // tile's rows past the end of the sequence read row N - 1, and the mask of that
  // always partial tile drops them.)
  uint32_t kin[CPW], vin[CPW];
#pragma unroll
  for (int j = 0; j < CPW; ++j) {
    kin[j] = (uint32_t)(krow[j] * D + kch[j]) * 2u;
    vin[j] = (uint32_t)(krow[j] * D + vch[j]) * 2u;
  }
  // HIL: key tile t is the curve's block t, and a copy's tile row is its
  // position in the block. Blocks entered in different states are transposes
  // and mirrors of one another, so each copy's byte offset from the block's
  // origin row is hA0 (state 0) or hA1 (transposed), with the K chunk in its low
  // bits, XORed with a uniform constant when the block is mirrored (both cell
  // coordinates XOR 7); the V chunk's offset differs from the K chunk's by the
  // XOR hX. Lane l also holds the local cells of local position l in a block
  // entered in state 0 (bits 0-5) and in a transposed one (bits 6-11), for the
  // lookups of the prologue.
  uint32_t hA0[CPW], hA1[CPW], hX[CPW];
  int e_lane = 0;
  if constexpr (HIL) {
    const uint32_t c0 = hilbert_local_walk((uint32_t)lane, 0);
    e_lane = (int)(c0 | hilbert_local_state(c0, 1) << 6);
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
      const uint32_t e = (uint32_t)__shfl(e_lane, krow[j]), c0 = e & 63u, c1 = e >> 6;
      const uint32_t kb = (uint32_t)kch[j] * 2u;
      hA0[j] = ((c0 >> 3) << a.lg | (c0 & 7u)) * (uint32_t)(D * 2) + kb;
      hA1[j] = ((c1 >> 3) << a.lg | (c1 & 7u)) * (uint32_t)(D * 2) + kb;
      hX[j] = kb ^ ((uint32_t)vch[j] * 2u);
    }
  }
  // (ioff: elements from this workgroup's first slice to the item's.)
  auto issue_tile = [&](int i, int stage, int64_t ioff = 0) {
    char *base = lds + stage * STAGE;
    const __bf16 *Kt = K + ioff, *Vt = V + ioff;
    uint32_t ko[CPW], vo[CPW];
    if constexpr (GATHER) {
      const int32_t *rows = idx_k(i);
#pragma unroll
      for (int j = 0; j < CPW; ++j) {
        const uint32_t r = (uint32_t)rows[krow[j]] * (uint32_t)(D * 2);
        ko[j] = r + (uint32_t)kch[j] * 2u;
        vo[j] = r + (uint32_t)vch[j] * 2u;
      }
    } else if constexpr (HIL) {
      // the block's origin row and entry state (uniform), into the slice base
      uint32_t ent;
      if (i < kBlkTab) {
        ent = __builtin_amdgcn_readfirstlane(reinterpret_cast<const uint32_t *>(lds + BLKT)[i]);
      } else {
        uint32_t bx, by, bst;
        hilbert_block((uint32_t)tile_of(i), a.lg, bx, by, bst);
        ent = (by << a.lg | bx) | bst;
      }
      Kt += (int64_t)(ent & ~3u) * D;
      Vt += (int64_t)(ent & ~3u) * D;
      const uint32_t mirror = (ent & 2u) ? (7u << a.lg | 7u) * (uint32_t)(D * 2) : 0u;
      const bool transposed = (ent & 1u) != 0;
#pragma unroll
      for (int j = 0; j < CPW; ++j) {
        ko[j] = (transposed ? hA1[j] : hA0[j]) ^ mirror;
        vo[j] = ko[j] ^ hX[j];
      }
    } else {
      const int k0 = tile_of(i) * BN;
      if (k0 + BN <= a.N) {
        Kt += (int64_t)k0 * D;
        Vt += (int64_t)k0 * D;
#pragma unroll
        for (int j = 0; j < CPW; ++j) {
          ko[j] = kin[j];
          vo[j] = vin[j];
        }
      } else {
#pragma unroll
        for (int j = 0; j < CPW; ++j) {
          const uint32_t r = (uint32_t)min(k0 + krow[j], a.N - 1) * (uint32_t)(D * 2);
          ko[j] = r + (uint32_t)kch[j] * 2u;
          vo[j] = r + (uint32_t)vch[j] * 2u;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < CPW; ++j)
      lds_dma16_at(Kt, ko[j], lds_addr(base + (j * NW + wave) * 1024));
#pragma unroll
    for (int j = 0; j < CPW; ++j)
      lds_dma16_at(Vt, vo[j], lds_addr(base + TILE + (j * NW + wave) * 1024));
  };
  // GATHER: the row indices of list entry i (one per lane of the first wave)
  // into its slot. RPB: every wave copies BN / NW of them. Positions past the end
  // of the sequence read entry N - 1.
  auto issue_idx = [&](int i) {
    if constexpr (GATHER) {
      if (wave == 0)
        lds_dma4(a.order + min(tile_of(i) * BN + lane, a.N - 1), lds_addr(lds + IDXK + (i & 3) * BN * 4));
    } else {
      constexpr int PER = BN / NW;   // ids per wave
      if (lane < PER)
        lds_dma4(a.order + min(tile_of(i) * BN + wave * PER + lane, a.N - 1),
                 lds_addr(lds + IDXK + (i & 3) * BN * 4 + wave * PER * 4));
    }
  };

  // LDS byte offsets (within a stage) of this lane's K operand reads for the
  // first 32-key block. The swizzle ignores row bit 5, so the second block's
  // reads sit exactly 32 rows further (an immediate offset of the LDS read).
  int kaddr[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int r = row_perm(col);
    kaddr[c] = r * D * 2 + (((half * NCH + c) ^ swz_k<D>(r)) * 16);
  }
  // V^T operand for (db, t): two transposing reads e = 0, 1. Lane i of 16-lane
  // group g points at row 16t + 8(g/2) + 4e + i/4, columns db*32 + 16(g%2) + 4(i%4).
  // The swizzle of those rows depends only on i/4, so (t, e) only add a constant
  // row offset (16t + 4e) * D * 2 bytes.
  const int g16 = lane >> 4, i16 = lane & 15;
  int vbase[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) {
    const int r = 8 * (g16 >> 1) + (i16 >> 2);
    const int cl = db * 32 + 16 * (g16 & 1) + 4 * (i16 & 3);
    vbase[db] = TILE + r * D * 2 + (((cl >> 3) ^ swz_v<D>(r)) * 16) + (cl & 7) * 2;
  }

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = f32x16{};
  float m_run = -__builtin_inff();  // running reference, in units of log2
  float l_run = 0.f;               // this lane's partial sum (its half of the keys)
  bool primed = false;             // every lane's m_run is finite (wave-uniform)
  // scores are multiplied by smul to reach log2 units (RPB: already scaled)
  const float smul = RPB ? 1.44269504088896340736f : a.scale_log2;

  // Prologue: the Q tile goes into stage 2 (which the third key tile fills
  // later), the first two key tiles into stages 0 and 1. Staging Q through LDS
  // keeps every global load of the kernel a tracked ring copy: a Q operand
  // loaded straight into registers would make the compiler wait for all copies
  // in flight before its first use in the loop.
  // HIL: wave 0 classifies this row's candidate key tiles (the key positions
  // any query of the tile may attend, per pattern) with the list builder's
  // classifier, one tile per lane. For the 1-D patterns the non-empty tiles of a
  // row are one run [t_lo, t_hi] and the full ones one run [f_lo, f_hi] inside
  // it, so the lists are "f_lo .. f_hi, then t_lo .. f_lo - 1, then f_hi + 1 ..
  // t_hi" (ascending within each, as the builder writes them); should a row
  // ever not have that shape, every tile of [t_lo, t_hi] runs masked instead.
  // It tabulates the curve blocks of the first list entries and hands the runs
  // to the other waves through LDS. Meanwhile every wave finds the row of its
  // own query (the output row).
  // HIL: the query tile's curve blocks (uniform) and the row of a position of
  // it in block c of the tile (c uniform; its local cell a cross-lane read).
  constexpr int QBLK = BM / 64;
  uint32_t bx[QBLK], by[QBLK], bst[QBLK];
  // (a tile reaching past the sequence, N = 64 < BM: its positions past the
  // end read the last row)
  int cmax = 0;
  if constexpr (HIL) {
    const uint32_t b0 = (uint32_t)(qt * BM) >> 6;
#pragma unroll
    for (int c = 0; c < QBLK; ++c) hilbert_block(b0 + c, a.lg, bx[c], by[c], bst[c]);
    cmax = ((a.N - 1) >> 6) - (int)b0;
  }
  auto row_in = [&](int c, int pos) {
    const int cc = min(c, cmax);
    uint32_t x = bx[0], y = by[0], st = bst[0];
#pragma unroll
    for (int k = 1; k < QBLK; ++k)
      if (cc == k) {
        x = bx[k];
        y = by[k];
        st = bst[k];
      }
    const uint32_t e = (uint32_t)__shfl(e_lane, min(pos, a.N - 1) & 63);
    const uint32_t cell = ((e >> (6 * (st & 1u))) & 63u) ^ ((st & 2u) ? 63u : 0u);
    return hilbert_block_row(x, y, cell, a.lg);
  };
  uint32_t my_row = 0;
  uint32_t qoff[LQ];
  if constexpr (HIL) {
    uint32_t *blkt = reinterpret_cast<uint32_t *>(lds + BLKT);
    int32_t *runs = reinterpret_cast<int32_t *>(lds + BLKT + kBlkTab * 4);
    if (wave == 0) {
      // candidate range (64-bit: window ends may pass 2^31 for parameters
      // near 2^30; the group quotients fit 32 bits)
      const int64_t i0 = (int64_t)qt * BM, i1 = min(i0 + BM - 1, (int64_t)P.N - 1);
      const int64_t w = P.p0;
      int64_t lo = 0, hi = P.N - 1;
      if (P.kind == HLA_HILBERT_WINDOW || P.kind == HLA_HILBERT_SHIFTED_WINDOW) {
        const uint32_t off = P.kind == HLA_HILBERT_WINDOW ? 0u : (uint32_t)(P.p0 - P.p1);
        const uint32_t ga = ((uint32_t)i0 + off) / (uint32_t)w, gb = ((uint32_t)i1 + off) / (uint32_t)w;
        lo = (int64_t)ga * w - off;
        hi = (int64_t)gb * w + w - 1 - off;
      } else if (P.kind == HLA_HILBERT_SLIDE) {
        lo = i0 - w;
        hi = i1 + w;
      } else if (P.kind == HLA_HILBERT_NEIGHBORHOOD) {
        lo = min(max(i0 - w / 2, (int64_t)0), (int64_t)P.N - w);
        hi = min(max(i1 - w / 2, (int64_t)0), (int64_t)P.N - w) + w - 1;
      }
      const int c_lo = (int)(max(lo, (int64_t)0) / BN), c_hi = (int)(min(hi, (int64_t)P.N - 1) / BN);
      int n_any = 0, n_full = 0, tl = 0x7fffffff, th = -1, fl = 0x7fffffff, fh = -1;
      for (int c0 = c_lo; c0 <= c_hi; c0 += 64) {
        const int kt = c0 + lane;
        const int cls = kt <= c_hi ? tile_class<true>(P, BM, BN, qt, kt) : 0;
        const uint64_t ba = __ballot(cls != 0), bf = __ballot(cls == 2);
        if (ba) {
          tl = min(tl, c0 + (int)__builtin_ctzll(ba));
          th = c0 + 63 - (int)__builtin_clzll(ba);
          n_any += __popcll(ba);
        }
        if (bf) {
          fl = min(fl, c0 + (int)__builtin_ctzll(bf));
          fh = c0 + 63 - (int)__builtin_clzll(bf);
          n_full += __popcll(bf);
        }
      }
      const bool one_run = n_any == th - tl + 1 && (n_full == 0 || n_full == fh - fl + 1);
      if (n_any > 0) {
        t_lo = tl;
        ntot = one_run ? n_any : th - tl + 1;
        if (one_run && n_full > 0) {
          nf = n_full;
          f_lo = fl;
          f_hi = fh;
        } else {
          f_lo = tl;
          f_hi = tl - 1;
        }
      }
      nf = __builtin_amdgcn_readfirstlane(nf);
      ntot = __builtin_amdgcn_readfirstlane(ntot);
      t_lo = __builtin_amdgcn_readfirstlane(t_lo);
      f_lo = __builtin_amdgcn_readfirstlane(f_lo);
      f_hi = __builtin_amdgcn_readfirstlane(f_hi);
      // the block table: origin row | entry state of each list entry's block
      for (int e = lane; e < min(ntot, kBlkTab); e += 64) {
        uint32_t x, y, st;
        hilbert_block((uint32_t)tile_of(e), a.lg, x, y, st);
        blkt[e] = (y << a.lg | x) | st;
      }
      if (lane == 0) {
        runs[0] = nf;
        runs[1] = ntot;
        runs[2] = t_lo;
        runs[3] = f_lo;
        runs[4] = f_hi;
      }
    }
    my_row = row_in(wave / 2, qpos);
    // (a copy's tile row lies in block (j * NW + wave) / CPR: it is a whole
    // multiple of 64 / CPR rows past the wave's first)
#pragma unroll
    for (int j = 0; j < LQ; ++j) {
      const int p = (j * NW + wave) * 64 + lane;
      const int r = p / CPR, cs = p % CPR;
      qoff[j] = row_in((j * NW + wave) / CPR, qt * BM + r) * (uint32_t)(D * 2) +
                (uint32_t)(cs ^ swz_q<D>(r)) * 16u;
    }
    // The first item's Q tile into stage 0 now (the first element of the copy
    // stream below), while wave 0 classifies; the barrier publishes wave 0's
    // LDS writes and leaves the copies in flight.
#pragma unroll
    for (int j = 0; j < LQ; ++j) lds_dma16_at(Q, qoff[j], lds_addr(lds + (j * NW + wave) * 1024));
    wait_then_barrier<63>();
    nf = __builtin_amdgcn_readfirstlane(runs[0]);
    ntot = __builtin_amdgcn_readfirstlane(runs[1]);
    t_lo = __builtin_amdgcn_readfirstlane(runs[2]);
    f_lo = __builtin_amdgcn_readfirstlane(runs[3]);
    f_hi = __builtin_amdgcn_readfirstlane(runs[4]);
  } else if constexpr (GATHER) {
    // Row indices of the Q tile and of the first three key tiles, first.
    if (wave == 0) {
#pragma unroll
      for (int c = 0; c < BM / 64; ++c)
        lds_dma4(a.order + min(qt * BM + 64 * c + lane, a.N - 1), lds_addr(lds + IDXQ + 256 * c));
    }
#pragma unroll
    for (int i = 0; i < 3; ++i)
      if (i < ntot) issue_idx(i);
    wait_then_barrier<0>();
  }
  // The Q tile's copies (Qs: the item's slice) into ring stage stg.
  // (HIL: from the slice base plus the copies' byte offsets qoff, found once.)
  auto issue_q = [&](const __bf16 *Qs, int stg) {
    char *base = lds + stg * STAGE;
#pragma unroll
    for (int j = 0; j < LQ; ++j) {
      if constexpr (HIL) {
        lds_dma16_at(Qs, qoff[j], lds_addr(base + (j * NW + wave) * 1024));
      } else {
        const int p = (j * NW + wave) * 64 + lane;
        const int r = p / CPR, cs = p % CPR;
        const int64_t row = GATHER ? (int64_t)idx_q[r] : (int64_t)min(qt * BM + r, a.N - 1);
        lds_dma16(Qs + row * D + (cs ^ swz_q<D>(r)) * 8, lds_addr(base + (j * NW + wave) * 1024));
      }
    }
  };
  if constexpr (!STREAM) {
    issue_q(Q, 2);
    if constexpr (RPB) {
      if (ntot > 0) issue_idx(0);
      if (ntot > 1) issue_idx(1);
    }
    if (ntot > 0) issue_tile(0, 0);
    if (ntot > 1) issue_tile(1, 1);
    if constexpr (RPB) {
      if (ntot > 2) issue_idx(2);
    }
  }
  // RPB: this lane's query cell (rq, cq) and bias base C + off(q), loaded after
  // the copies; one wait the compiler sees then covers it and them. Then the
  // workgroup's query box: each wave's, combined through LDS.
  int32_t rpb_base = 0, rq = 0, cq = 0, qr0 = 0, qr1 = 0, qc0 = 0, qc1 = 0;
  const float *rpb_h = nullptr;
  if constexpr (RPB) {
    const int32_t g = a.order[min(qpos, a.N - 1)];
    const int32_t Wg = P.W;
    rq = (int32_t)fdiv((uint32_t)g, P.wdiv);
    cq = g - rq * Wg;
    rpb_base = (P.H - 1) * (2 * Wg - 1) + (Wg - 1) + g + (Wg - 1) * rq;
    rpb_h = a.rpb + (int64_t)(bh % a.heads) * (2 * P.H - 1) * (2 * Wg - 1);
    wait_vmem_all();
    int4 box = wave_box(rq, cq);
    if (lane == 0) reinterpret_cast<int4 *>(lds + QBOX)[wave] = box;
    wait_then_barrier<0>();
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const int4 b = reinterpret_cast<const int4 *>(lds + QBOX)[w];
      box = int4{min(box.x, b.x), max(box.y, b.y), min(box.z, b.z), max(box.w, b.w)};
    }
    qr0 = __builtin_amdgcn_readfirstlane(box.x);
    qr1 = __builtin_amdgcn_readfirstlane(box.y);
    qc0 = __builtin_amdgcn_readfirstlane(box.z);
    qc1 = __builtin_amdgcn_readfirstlane(box.w);
  } else if constexpr (!STREAM) {
    // Q and the first key tile are in; the second may still be in flight.
    if (ntot > 1) wait_then_barrier<LPT>();
    else wait_then_barrier<0>();
  }
  // This lane's Q operand, from the Q tile in ring stage stg.
  bf16x8 qop[NCH];
  auto load_q = [&](int stg) {
    const int r = wave * 32 + col;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
      qop[c] = *reinterpret_cast<const bf16x8 *>(lds + stg * STAGE + r * D * 2 +
                                                 (((half * NCH + c) ^ swz_q<D>(r)) * 16));
  };
  if constexpr (!STREAM) load_q(2);

  // RPB: the bias window of list entry j, issued by one wave: the table entries
  // that this workgroup's queries and entry j's keys can address - the rectangle
  // of cell offsets spanned by the query box and the key tile's box - copied
  // into window buffer j % 2, its parameters {dr0, dc0, wc, n} into slot j % 4,
  // and each key's term rk * wc + ck (one key per lane) into that slot's terms.
  // A tile whose window exceeds kWinCap entries gets n = 0 and reads the table
  // directly. Every table index copied lies in the table: both boxes are inside
  // the grid.
  auto issue_window = [&](int j) {
    const int32_t id = idx_k(j)[lane];
    const int32_t rk = (int32_t)fdiv((uint32_t)id, P.wdiv);
    const int4 kbox = wave_box(rk, id - rk * P.W);
    const int32_t kr0 = __builtin_amdgcn_readfirstlane(kbox.x);
    const int32_t kr1 = __builtin_amdgcn_readfirstlane(kbox.y);
    const int32_t kc0 = __builtin_amdgcn_readfirstlane(kbox.z);
    const int32_t kc1 = __builtin_amdgcn_readfirstlane(kbox.w);
    const int32_t dr0 = qr0 - kr1, dc0 = qc0 - kc1;
    const int32_t wc = qc1 - kc0 - dc0 + 1, n = (qr1 - kr0 - dr0 + 1) * wc;
    const bool fits = n <= kWinCap;
    if (lane == 0) *reinterpret_cast<int4 *>(lds + WINP + (j & 3) * 16) = int4{dr0, dc0, wc, fits ? n : 0};
    if (fits) {
      reinterpret_cast<int32_t *>(lds + WINB + (j & 3) * BN * 4)[lane] = id + rk * (wc - P.W);
      // entry f of the window is offset row f / wc, column f % wc (the row from
      // a float quotient: exact, as f < 2^10 puts the fraction >= 2^-11 away
      // from an integer)
      const float inv = 1.f / (float)wc;
      const int32_t pitch = 2 * P.W - 1, last = (2 * P.H - 1) * pitch - 1;
      for (int c = 0; c * 64 < n; ++c) {
        const int32_t f = min(64 * c + lane, n - 1);
        const int32_t i = (int32_t)(((float)f + 0.5f) * inv);
        const int32_t jj = f - i * wc;
        // (clamped as a guard: the boxes already keep it inside the table)
        const int32_t e = min(max((dr0 + i + P.H - 1) * pitch + (dc0 + jj + P.W - 1), 0), last);
        lds_dma4(rpb_h + e, lds_addr(lds + WIN + (j & 1) * kWinCap * 4 + 256 * c));
      }
    }
  };
  if constexpr (RPB) {
    // entry 0's window, complete and visible before the loop
    if (ntot > 0 && wave == 0) issue_window(0);
    wait_then_barrier<0>();
  }

  // The math of one key tile staged at st (list entry it): S^T, (mask), online
  // softmax and O^T += V^T P^T.
  auto tile_math = [&](const char *st, int it, auto masked) {
    // S^T for the two 32-key blocks (independent accumulators interleaved), the
    // RPB bias and the mask: the tile's scores, this lane's 32 of them.
    auto scores = [&](f32x16 (&s)[2]) {
      s[0] = f32x16{};
      s[1] = f32x16{};
#pragma unroll
      for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const bf16x8 kop = *reinterpret_cast<const bf16x8 *>(st + kaddr[c] + kb * 32 * D * 2);
          s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop, qop[c], s[kb], 0, 0, 0);
        }
      // RPB: scores in natural units plus the bias, s = scale * <q, k> + bias,
      // from the tile's staged window (entry (rq - rk - dr0) * wc + (cq - ck -
      // dc0)) or, for a tile whose window did not fit, from the table.
      if constexpr (RPB) {
        const int32_t *kid = idx_k(it);
        const int4 pw = *reinterpret_cast<const int4 *>(lds + WINP + (it & 3) * 16);
        const int32_t w_dr0 = __builtin_amdgcn_readfirstlane(pw.x);
        const int32_t w_dc0 = __builtin_amdgcn_readfirstlane(pw.y);
        const int32_t w_wc = __builtin_amdgcn_readfirstlane(pw.z);
        const int32_t w_n = __builtin_amdgcn_readfirstlane(pw.w);
        float bias[2][16];
        if (w_n != 0) {
          const float *win = reinterpret_cast<const float *>(lds + WIN + (it & 1) * kWinCap * 4);
          const int32_t *term = reinterpret_cast<const int32_t *>(lds + WINB + (it & 3) * BN * 4);
          const int32_t aq = (rq - w_dr0) * w_wc + (cq - w_dc0);
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int g = 0; g < 2; ++g) {
              const int4 *tk = reinterpret_cast<const int4 *>(term + kb * 32 + 16 * g + 8 * half);
              const int4 lo = tk[0], hi = tk[1];
              const int32_t bk[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
              for (int e = 0; e < 8; ++e) bias[kb][8 * g + e] = win[aq - bk[e]];
            }
        } else {
          // all 32 bias loads first, so that they are in flight together
          const int32_t Wm1 = P.W - 1;
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int g = 0; g < 2; ++g) {
              const int4 *ids = reinterpret_cast<const int4 *>(kid + kb * 32 + 16 * g + 8 * half);
              const int4 lo = ids[0], hi = ids[1];
              const int32_t gk[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                const int32_t koff = gk[e] + Wm1 * (int32_t)fdiv((uint32_t)gk[e], P.wdiv);
                bias[kb][8 * g + e] = rpb_h[rpb_base - koff];
              }
            }
        }
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int v = 0; v < 16; ++v) s[kb][v] = __builtin_fmaf(s[kb][v], a.scale, bias[kb][v]);
      }
      if constexpr (decltype(masked)::value) mask_blocks<2>(s, R, P, tile_of(it) * BN + 8 * half);
    };
    // Weights p = 2^(s * smul - m) in place of the scores; returns l0 plus this
    // lane's sum of them (two running sums, one per key block, the first seeded
    // with l0).
    auto weights = [&](f32x16 (&s)[2], float m, float l0) {
      float la = l0, lb = 0.f;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[0][v], smul, -m));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[1][v], smul, -m));
        la += p0;
        lb += p1;
        s[0][v] = p0;
        s[1][v] = p1;
      }
      return la + lb;
    };

    // Online softmax in the log2 domain with a lazily moved reference m_run
    // (O and l always share it). Once every row of the wave has a finite
    // reference, a tile first takes its weights against the reference as it
    // stands, with no row max at all: weights up to 2^32 are harmless (fp32
    // accumulators, bf16 operands), and since they and l_run are >= 0 the new
    // running sum bounds each of them, so one compare of it (NaN and inf fail it
    // too) validates the tile. Only when some row's sum fails does the tile
    // fall back: its scores are recomputed from LDS and it takes the max path,
    // l_run being untouched until the tile is accepted. (Straight-line code
    // rather than a retry loop: with a loop, the compiler kept O in two register
    // sets and copied it on every tile.)
    f32x16 s[2];
    scores(s);
    bool slow = !primed;
    float ln = 0.f;
    if (primed) {
      ln = weights(s, m_run, l_run);
      if (__ballot(!(ln <= kFastBound))) {
        slow = true;
        // (the memory clobber makes the K operand reads happen again instead of
        // keeping the first ones in registers across the weights)
        asm volatile("" ::: "memory");
        scores(s);
      }
    }
    if (slow) {
      // Max path: the reference moves only when a row's tile max exceeds it by
      // more than kRescaleSlack, so the O / l rescale stays rare.
      float mq[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x16 &sv = s[g >> 1];
        const int o = 8 * (g & 1);
        mq[g] = fmaxf(fmaxf(fmaxf(sv[o], sv[o + 1]), fmaxf(sv[o + 2], sv[o + 3])),
                      fmaxf(fmaxf(sv[o + 4], sv[o + 5]), fmaxf(sv[o + 6], sv[o + 7])));
      }
      const float mx = xhalf_max(fmaxf(fmaxf(mq[0], mq[1]), fmaxf(mq[2], mq[3])));
      const float mt = mx * smul;
      const bool grow = mt > m_run + kRescaleSlack;
      if (__ballot(grow)) {
        const float m_new = grow ? mt : m_run;
        // A row whose reference is still -inf has seen no allowed key: its O
        // and l are exactly 0. So when no row of the wave has a finite
        // reference (a row's first tile), the rescale is skipped.
        if (__ballot(m_run != -__builtin_inff())) {
          // 1 where unchanged; a row with no allowed key yet has nothing to rescale
          const float alpha = m_new == -__builtin_inff() ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
          l_run *= alpha;
#pragma unroll
          for (int db = 0; db < NDB; ++db) oacc[db] *= alpha;
        }
        m_run = m_new;
      }
      ln = weights(s, m_run == -__builtin_inff() ? 0.f : m_run, l_run);
      primed = !__ballot(m_run == -__builtin_inff());
    }
    l_run = ln;
    // Row sums above are fp32 sums of the unrounded weights; P goes to the PV
    // product rounded to bf16.
    bf16x8 pop[4];
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int e = 0; e < 8; ++e) pop[g][e] = (__bf16)s[g >> 1][8 * (g & 1) + e];

    // O^T += V^T P^T over four 16-key steps, d blocks interleaved; V^T
    // operands read with the transposing LDS read right before use.
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const bf16x8 vop = lds_read_tr16x2(st + vbase[db] + (16 * t) * D * 2, D * 2);
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop, pop[t], oacc[db], 0, 0, 0);
      }
  };

  // One key tile: wait for its copies, refill the ring, then S^T, (mask),
  // online softmax and O^T += V^T P^T. MASKED is a compile-time flag, so full
  // and partial tiles run separate loop bodies and the unmasked path carries no
  // mask code at all.
  int stage = 0;
  auto step = [&](int it, auto masked) {
    // Wait for this wave's copies of tile `it`; the copies of tile it + 1 (the
    // only one issued after it) may stay in flight.
    // RPB: after tile it's window come tile it + 1's copies and entry it + 2's
    // indices.
    if (RPB && it + 2 < ntot) wait_then_barrier<LPT + 1>();
    else if (it + 1 < ntot) wait_then_barrier<LPT>();
    else wait_then_barrier<0>();
    // The stage refilled next was last read in iteration it - 1, which every
    // wave has finished (it is behind the barrier above).
    const int nstage = stage == 0 ? 2 : stage - 1;  // (it + 2) % 3
    // (GATHER: the indices of entry it + 2 arrived with the wait above, those of
    // it + 3 go out first.)
    if constexpr (GATHER) {
      if (it + 3 < ntot) issue_idx(it + 3);
    }
    if constexpr (!RPB) {
      if (it + 2 < ntot) issue_tile(it + 2, nstage);
    }
    const char *st = lds + stage * STAGE;
    stage = stage == 2 ? 0 : stage + 1;

    tile_math(st, it, masked);
    // RPB: at the end of the step, entry it + 1's window (its indices arrived
    // before this step's barrier), then the ring refill (stage (it + 2) % 3 held
    // tile it - 1, which every wave finished before this step's barrier), then
    // entry it + 3's indices (slot (it + 3) % 4 last held entry it - 1's).
    if constexpr (RPB) {
      if (it + 1 < ntot && wave == (it + 1) % NW) issue_window(it + 1);
      if (it + 2 < ntot) issue_tile(it + 2, nstage);
      if (it + 3 < ntot) issue_idx(it + 3);
    }
  };
  // Epilogue: normalise and store the rows straight from the accumulators. Lane
  // (col, half) holds, per d block and 8-row group a, the four values
  // d = 8a + 4half + 0..3 of query col; one exchange with lane col ^ 32 per pair
  // of groups gives each lane eight consecutive values (16 bytes) to store.
  // (sl: the item's slice, bhh: its head index)
  auto store_rows = [&](int64_t sl, int bhh) {
    const float l_tot = xhalf_sum(l_run);
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    // (queries past the end of the sequence, in a ragged last query tile, take part
    // in the exchanges but store nothing)
    const bool live = qpos < a.N;
    const int64_t out_row = GATHER ? (int64_t)idx_q[wave * 32 + col] : HIL ? (int64_t)my_row : (int64_t)qpos;
    __bf16 *orow = static_cast<__bf16 *>(a.out) + sl + out_row * D;
  #pragma unroll
    for (int db = 0; db < NDB; ++db)
  #pragma unroll
      for (int pr = 0; pr < 2; ++pr) {
        bf16x4 x0, x1;
  #pragma unroll
        for (int b = 0; b < 4; ++b) {
          x0[b] = (__bf16)(oacc[db][8 * pr + b] * inv);
          x1[b] = (__bf16)(oacc[db][8 * pr + 4 + b] * inv);
        }
        const uint2 u0 = __builtin_bit_cast(uint2, x0), u1 = __builtin_bit_cast(uint2, x1);
        // half 0 keeps group 2pr and receives the partner's part of it; half 1
        // keeps group 2pr + 1 and receives the partner's part of that.
        const uint2 send = half ? u0 : u1;
        uint2 recv;
        recv.x = __shfl_xor(send.x, 32);
        recv.y = __shfl_xor(send.y, 32);
        const uint4 row = half ? uint4{recv.x, recv.y, u1.x, u1.y} : uint4{u0.x, u0.y, recv.x, recv.y};
        if (live) *reinterpret_cast<uint4 *>(orow + db * 32 + 16 * pr + 8 * half) = row;
      }
    if (a.lse && half == 0 && live) {
      const float ln2 = 0.69314718055994530942f;
      a.lse[(int64_t)bhh * a.N + out_row] =
          l_tot > 0.f ? (m_run + __builtin_amdgcn_logf(l_tot)) * ln2 : -__builtin_inff();
    }
  };

  if constexpr (STREAM) {
    // The items as one stream of ring copies: item h's Q tile, then its list's
    // key tiles, then item h + 1's. Element e goes into stage e % 3 once every
    // wave has read element e - 3, so the next item's Q tile and first key tile
    // are copied during the current item's last two tiles, and the workgroup's
    // tile list (HIL: its classification, block table and rows) serves every
    // item. The previous item's rows are stored after the next item's first
    // wait, so that wait never waits for stores.
    const int64_t ND = (int64_t)a.N * D;
    if (ntot == 0) {
      wait_vmem_all();  // the unused Q copies land before the workgroup ends
      for (int h = 0; h < nitems; ++h) store_rows(slice + h * ND, bh + h);
      return;
    }
    // Element e + 2 goes out when element e is read: in stage (s + 2) % 3 for
    // the element read from stage s. Within an item that is its entry it + 2;
    // the item's last two entries hand over to the next item's Q tile and its
    // entry 0.
    // (element 0, the first item's Q tile, went out in the prologue)
    issue_tile(0, 1);
    if (ntot > 1) issue_tile(1, 2);
    else if (nitems > 1) issue_q(Q + ND, 2);
    int h = 0, cstage = 0;  // item, stage of the element read next
    int64_t ioff = 0;       // elements from the first item's slice to item h's
    // List entry it of item h: wait for its copies (the one element issued
    // after it may stay in flight: the item's next entry, or the next item's
    // Q tile), refill the ring, the math.
    auto hil_step = [&](int it, auto masked) {
      const int nst = cstage == 0 ? 2 : cstage - 1;
      if (it + 2 < ntot) {
        if (h > 0 && it == 0) wait_then_barrier<63>();  // entry 0 arrived before the item began
        else wait_then_barrier<LPT>();
        issue_tile(it + 2, nst, ioff);
      } else {
        if (h > 0 && it == 0) wait_then_barrier<63>();
        else if (it + 1 < ntot) wait_then_barrier<LPT>();
        else if (h + 1 < nitems) wait_then_barrier<LQ>();
        else wait_then_barrier<0>();
        if (h + 1 < nitems) {
          if (it + 2 == ntot) issue_q(Q + ioff + ND, nst);
          else issue_tile(0, nst, ioff + ND);
        }
      }
      const char *st = lds + cstage * STAGE;
      cstage = cstage == 2 ? 0 : cstage + 1;
      tile_math(st, it, masked);
    };
    for (h = 0; h < nitems; ++h, ioff += ND) {
      // the item's Q tile and list entry 0 are in (at the first item the
      // third element may still be in flight; later, nothing was issued after
      // them); then the stage of the previous item's last entry takes the
      // element after the item's entry 0
      if (h == 0) {
        if (ntot > 1) wait_then_barrier<LPT>();
        else if (nitems > 1) wait_then_barrier<LQ>();
        else wait_then_barrier<0>();
      } else {
        wait_then_barrier<0>();
        const int nst = cstage == 0 ? 2 : cstage - 1;
        if (ntot > 1) issue_tile(1, nst, ioff);
        else if (h + 1 < nitems) issue_q(Q + ioff + ND, nst);
      }
      // Waves of the workgroup that has more items left issue first: a CU's
      // workgroups start together, and the arbiter would otherwise favour the
      // older one, leaving the younger to finish alone.
      {
        const int left = (nitems - h) >> 1;
        if (left >= 3) __builtin_amdgcn_s_setprio(3);
        else if (left == 2) __builtin_amdgcn_s_setprio(2);
        else if (left == 1) __builtin_amdgcn_s_setprio(1);
        else __builtin_amdgcn_s_setprio(0);
      }
      if (h > 0) {
        store_rows(slice + ioff - ND, bh + h - 1);
#pragma unroll
        for (int db = 0; db < NDB; ++db) oacc[db] = f32x16{};
        m_run = -__builtin_inff();
        l_run = 0.f;
        primed = false;
      }
      load_q(cstage);
      cstage = cstage == 2 ? 0 : cstage + 1;
      for (int it = 0; it < nf; ++it) hil_step(it, std::false_type{});
      for (int it = nf; it < ntot; ++it) hil_step(it, std::true_type{});
    }
    store_rows(slice + (nitems - 1) * ND, bh + nitems - 1);
  } else {
    for (int it = 0; it < nf; ++it) step(it, std::false_type{});
    for (int it = nf; it < ntot; ++it) step(it, std::true_type{});
    store_rows(slice, bh);
  }
}

// Heads per workgroup of the one-launch mode. A workgroup's set-up (the tile
// classification, the block table and rows, the first copies' latency) is paid
// once for all its heads, while too few workgroups leave resident slots empty
// and an extra partial round lengthens the tail. With `slots` = CUs x the
// kernel's resident workgroups per CU, h* = B*heads*query tiles / slots heads
// per workgroup is exactly one round: take the smallest count >= h* that
// divides B*heads (equal groups; the grid's contiguous shares, one per XCD,
// then carry equal work), within kHeadsWork key tiles of work per workgroup
// (the row's key span in tiles, from the pattern) and 8 heads; else the
// largest dividing count within that cap. HLA_ATTN_HEADS_PER_WORKGROUP
// (1 .. 64) overrides it. (The plain mode, whose set-up is only its list reads
// and first copies, gained at most 7% from several heads per workgroup and
// lost at some counts; it keeps one.)
constexpr int kHeadsWork = 48;
int heads_per_workgroup(const AttnArgs &a, int BM, int per_cu) {
  if (const char *env = std::getenv("HLA_ATTN_HEADS_PER_WORKGROUP")) {
    const int h = std::atoi(env);
    if (h >= 1 && h <= 64) return h;
  }
  const int cus = device_cu_count();
  // key positions a query may reach: the window, band or neighbourhood
  const int64_t span = a.pat.kind == HLA_HILBERT_SLIDE ? 2 * (int64_t)a.pat.p0 + 1 : (int64_t)a.pat.p0;
  const int64_t tiles = (std::min<int64_t>(span, a.N) + BM + BN - 1) / BN;
  const int cap = (int)std::max<int64_t>(1, std::min<int64_t>(std::min<int64_t>(8, kHeadsWork / tiles), a.BH));
  const int64_t slots = (int64_t)cus * std::max(per_cu, 1);
  const int64_t items = (int64_t)a.BH * a.n_qtiles;
  if (items <= slots) return 1;
  for (int d = 1; d <= cap; ++d)  // smallest dividing count that fits one round
    if (a.BH % d == 0 && (int64_t)(a.BH / d) * a.n_qtiles <= slots) return d;
  for (int d = cap; d > 1; --d)   // else the largest dividing count within the cap
    if (a.BH % d == 0) return d;
  return 1;
}

template <int D, int NW>
hipError_t launch(const AttnArgs &a_in, hipStream_t s) {
  AttnArgs a = a_in;
  if (a.mode == ATTN_HILBERT) {
    // resident workgroups per CU for this kernel, read once per instantiation
    static int per_cu = 0;
    if (!per_cu) {
      int n = 0;
      per_cu = hipOccupancyMaxActiveBlocksPerMultiprocessor(
                   &n, reinterpret_cast<const void *>(&attn_fwd_bf16<D, NW, ATTN_HILBERT>), 64 * NW, 0) ==
                           hipSuccess && n > 0
                   ? n : 1;
    }
    const int h = heads_per_workgroup(a, 32 * NW, per_cu);
    a.hgroups = (a.BH + h - 1) / h;  // groups of ceil or floor of BH / hgroups heads
  } else {
    a.hgroups = a.BH;
  }
  const int64_t blocks = (int64_t)a.hgroups * a.n_qtiles;
  if (a.mode == ATTN_GATHER)
    hipLaunchKernelGGL((attn_fwd_bf16<D, NW, ATTN_GATHER>), dim3((uint32_t)blocks), dim3(64 * NW), 0, s, a);
  else if (a.mode == ATTN_HILBERT)
    hipLaunchKernelGGL((attn_fwd_bf16<D, NW, ATTN_HILBERT>), dim3((uint32_t)blocks), dim3(64 * NW), 0, s, a);
  else if (a.mode == ATTN_RPB)
    hipLaunchKernelGGL((attn_fwd_bf16<D, NW, ATTN_RPB>), dim3((uint32_t)blocks), dim3(64 * NW), 0, s, a);
  else
    hipLaunchKernelGGL((attn_fwd_bf16<D, NW, ATTN_PLAIN>), dim3((uint32_t)blocks), dim3(64 * NW), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bf16(const AttnArgs &a, int d, int tile_m, int tile_n,
                            hipStream_t s) {
  if (tile_n != BN) return hipErrorInvalidValue;
  if (d == 64 && tile_m == 128) return launch<64, 4>(a, s);
  if (d == 64 && tile_m == 64) return launch<64, 2>(a, s);
  if (d == 32 && tile_m == 128) return launch<32, 4>(a, s);
  if (d == 32 && tile_m == 64) return launch<32, 2>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace hla
