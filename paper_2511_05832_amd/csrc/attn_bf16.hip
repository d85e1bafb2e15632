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
//                  from LDS, B = the wave's Q (kept in registers all kernel).
//   softmax        lane l owns query l%32; its 32 scores of the tile sit in its
//                  own accumulators (16 per key block, the other half of the keys
//                  in lane l^32), so row max / sum need one cross-half exchange.
//   O^T += V^T P^T (d x queries): D/32 blocks x 4 MFMAs. A = V^T from LDS,
//                  B = P straight from the S^T accumulators (see below).
//
// Register-resident P. The accumulator of a 32x32 MFMA holds, in lane
// (col = l%32, half = l/32) and slot v, row 8*(v/4) + 4*half + v%4. The K rows
// fed to S^T are permuted (key_of_row) so that accumulator slot v of lane half
// `half` is key 16*(v/8) + 8*half + v%8 of the block: eight consecutive keys per
// run, which is exactly the B-operand layout of the PV MFMA over 16 keys. So P
// goes from fp32 accumulators to bf16 operands in place, with no LDS trip.
// The contraction over d in S^T is likewise permuted (lane half `half` holds d
// in [half*D/2, (half+1)*D/2)), so each lane loads its Q slice as one
// contiguous run.
//
// LDS per stage: K as [BN][D+8] and V transposed as [D][BN+8] (bf16, padded so
// the 16-byte MFMA operand reads of 32 lanes hit distinct banks); two stages,
// filled from registers that were loaded two tiles ahead, one barrier per tile.
// Tile-list entries are read with scalar loads, so waiting for one never waits
// for the K/V vector loads in flight. Accumulators live in ordinary VGPRs (the
// library is built with the VGPR form of MFMA), so the softmax touches them
// without copies.
//
// Masking (partial tiles only). For the 1-D Hilbert patterns each query's
// allowed keys are one interval [lo, hi] computed once per lane; for the
// row-major patterns they are one rectangle of grid cells. Masked scores are
// -inf before the row max; a query with no allowed key so far keeps m = -inf and
// contributes exactly zero.
//
// Grid: one workgroup per (b*h, query tile), remapped so each XCD (workgroups
// are dealt round-robin to the 8 XCDs) receives a contiguous range of query
// tiles: neighbouring tiles share key/value tiles (a window is two query tiles;
// a band overlaps its neighbour almost entirely), and the reuse stays in one
// XCD's L2.
#include "hla_internal.h"

namespace hla {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int BN = 64;
constexpr int VS = BN + 8;  // row stride of transposed V in LDS (elements)
constexpr float kRescaleSlack = 8.f;  // log2 units the softmax reference may lag the max

// Combine a value of lane l with lane l ^ 32 (the other half of a query's keys).
__device__ __forceinline__ float xhalf_max(float x) { return fmaxf(x, __shfl_xor(x, 32)); }
__device__ __forceinline__ float xhalf_sum(float x) { return x + __shfl_xor(x, 32); }

__device__ __forceinline__ int key_of_row(int i) {
  // accumulator row i = 8a + 4g + b  ->  key 16(a/2) + 8g + 4(a%2) + b
  const int a = i >> 3, g = (i >> 2) & 1, b = i & 3;
  return 16 * (a >> 1) + 8 * g + 4 * (a & 1) + b;
}

__device__ __forceinline__ int xcd_remap(int bid, int total) {
  const int per = total >> 3, rem = total & 7;
  const int xcd = bid & 7, slot = bid >> 3;
  return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

__device__ __forceinline__ int clampi(int x, int lo, int hi) { return min(max(x, lo), hi); }

// Scalar (SMEM) load of a wave-uniform int through the constant address space.
__device__ __forceinline__ int sload(const int32_t *p) {
  return *(const __attribute__((address_space(4))) int32_t *)p;
}

// K tile rows are copied as 16-byte units; V is read as (2 d x 8 keys) units of
// eight 4-byte loads and written transposed (8 keys contiguous per d) after a
// byte permute, so the PV operand reads are 16 contiguous bytes.
template <int D, int NT>
__device__ __forceinline__ void load_tile(u32x4 (&k)[(BN * D / 8 + NT - 1) / NT],
                                          uint32_t (&v)[((D / 2) * (BN / 8) + NT - 1) / NT][8],
                                          const __bf16 *K, const __bf16 *V, int kt, int tid) {
  constexpr int KUNITS = BN * D / 8, KPT = (KUNITS + NT - 1) / NT;
  constexpr int VUNITS = (D / 2) * (BN / 8), VPT = (VUNITS + NT - 1) / NT;
  const __bf16 *Kt = K + (int64_t)kt * BN * D;
  const __bf16 *Vt = V + (int64_t)kt * BN * D;
#pragma unroll
  for (int u = 0; u < KPT; ++u) {
    const int id = tid + u * NT;
    if (KUNITS % NT == 0 || id < KUNITS)
      k[u] = *reinterpret_cast<const u32x4 *>(Kt + (id / (D / 8)) * D + (id % (D / 8)) * 8);
  }
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    const int id = tid + u * NT;
    if (VUNITS % NT == 0 || id < VUNITS) {
      const int dp = id % (D / 2), kg = id / (D / 2);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        v[u][j] = *reinterpret_cast<const uint32_t *>(Vt + (kg * 8 + j) * D + 2 * dp);
    }
  }
}

template <int D, int NT>
__device__ __forceinline__ void store_tile(const u32x4 (&k)[(BN * D / 8 + NT - 1) / NT],
                                           const uint32_t (&v)[((D / 2) * (BN / 8) + NT - 1) / NT][8],
                                           __bf16 *Ks, __bf16 *Vs, int tid) {
  constexpr int KS = D + 8;
  constexpr int KUNITS = BN * D / 8, KPT = (KUNITS + NT - 1) / NT;
  constexpr int VUNITS = (D / 2) * (BN / 8), VPT = (VUNITS + NT - 1) / NT;
#pragma unroll
  for (int u = 0; u < KPT; ++u) {
    const int id = tid + u * NT;
    if (KUNITS % NT == 0 || id < KUNITS)
      *reinterpret_cast<u32x4 *>(Ks + (id / (D / 8)) * KS + (id % (D / 8)) * 8) = k[u];
  }
#pragma unroll
  for (int u = 0; u < VPT; ++u) {
    const int id = tid + u * NT;
    if (VUNITS % NT == 0 || id < VUNITS) {
      const int dp = id % (D / 2), kg = id / (D / 2);
      u32x4 lo4, hi4;  // d = 2dp (low halves) and d = 2dp+1 (high halves), 8 keys each
      lo4.x = __builtin_amdgcn_perm(v[u][1], v[u][0], 0x05040100u);
      lo4.y = __builtin_amdgcn_perm(v[u][3], v[u][2], 0x05040100u);
      lo4.z = __builtin_amdgcn_perm(v[u][5], v[u][4], 0x05040100u);
      lo4.w = __builtin_amdgcn_perm(v[u][7], v[u][6], 0x05040100u);
      hi4.x = __builtin_amdgcn_perm(v[u][1], v[u][0], 0x07060302u);
      hi4.y = __builtin_amdgcn_perm(v[u][3], v[u][2], 0x07060302u);
      hi4.z = __builtin_amdgcn_perm(v[u][5], v[u][4], 0x07060302u);
      hi4.w = __builtin_amdgcn_perm(v[u][7], v[u][6], 0x07060302u);
      *reinterpret_cast<u32x4 *>(Vs + (2 * dp) * VS + kg * 8) = lo4;
      *reinterpret_cast<u32x4 *>(Vs + (2 * dp + 1) * VS + kg * 8) = hi4;
    }
  }
}

template <int D, int NW>
__global__ void __launch_bounds__(64 * NW)
    attn_fwd_bf16(AttnArgs a) {
  constexpr int BM = 32 * NW;
  constexpr int NT = 64 * NW;
  constexpr int KS = D + 8;          // row stride of K in LDS (elements)
  constexpr int STAGE = BN * KS + D * VS;
  constexpr int NCH = D / 16;        // MFMA steps over d for S^T
  constexpr int NDB = D / 32;        // d blocks of O^T
  constexpr int KUNITS = BN * D / 8; // 16-byte units of a K tile
  constexpr int KPT = (KUNITS + NT - 1) / NT;
  constexpr int VUNITS = (D / 2) * (BN / 8);  // (2 d x 8 keys) units of a V tile
  constexpr int VPT = (VUNITS + NT - 1) / NT;

  __shared__ __attribute__((aligned(16))) __bf16 lds[2 * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, half = lane >> 5;

  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = logical / a.n_qtiles;
  const int qt = logical - bh * a.n_qtiles;
  const int q0 = qt * BM;
  const int64_t slice = (int64_t)bh * a.N * D;
  const __bf16 *Q = static_cast<const __bf16 *>(a.q) + slice;
  const __bf16 *K = static_cast<const __bf16 *>(a.k) + slice;
  const __bf16 *V = static_cast<const __bf16 *>(a.v) + slice;

  // This lane's query and its Q operand (d = half*D/2 + 8c + s for step c).
  const int qpos = q0 + wave * 32 + col;
  bf16x8 qop[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
    qop[c] = *reinterpret_cast<const bf16x8 *>(Q + (int64_t)qpos * D + half * (D / 2) + 8 * c);

  // Allowed-key region of this query (used on partial tiles only).
  const PatternArgs &P = a.pat;
  const bool one_d = P.kind == HLA_HILBERT_WINDOW || P.kind == HLA_HILBERT_SLIDE ||
                     P.kind == HLA_HILBERT_NEIGHBORHOOD || P.kind == HLA_HILBERT_SHIFTED_WINDOW;
  const bool row_runs = (P.W & 7) == 0;
  int lo = 0, hi = 0, rlo = 0, rhi = 0, clo = 0, chi = 0;
  if (P.kind == HLA_HILBERT_WINDOW) {
    lo = (qpos / P.p0) * P.p0;
    hi = lo + P.p0 - 1;
  } else if (P.kind == HLA_HILBERT_SLIDE) {
    lo = qpos - P.p0;
    hi = qpos + P.p0;
  } else if (P.kind == HLA_HILBERT_NEIGHBORHOOD) {
    lo = clampi(qpos - P.p0 / 2, 0, P.N - P.p0);
    hi = lo + P.p0 - 1;
  } else if (P.kind == HLA_HILBERT_SHIFTED_WINDOW) {
    const int g = (qpos + P.p0 - P.p1) / P.p0;
    lo = g * P.p0 - P.p0 + P.p1;
    hi = lo + P.p0 - 1;
  } else {
    const int r = (int)fdiv((uint32_t)qpos, P.wdiv), c = qpos - r * P.W;
    if (P.kind == HLA_ROWMAJOR_WINDOW) {
      rlo = (r / P.p0) * P.p0; rhi = rlo + P.p0 - 1;
      clo = (c / P.p1) * P.p1; chi = clo + P.p1 - 1;
    } else if (P.kind == HLA_ROWMAJOR_SLIDE) {
      rlo = r - P.p0; rhi = r + P.p0;
      clo = c - P.p1; chi = c + P.p1;
    } else {
      rlo = clampi(r - P.p0 / 2, 0, P.H - P.p0); rhi = rlo + P.p0 - 1;
      clo = clampi(c - P.p1 / 2, 0, P.W - P.p1); chi = clo + P.p1 - 1;
    }
  }

  // Tile-list reads are uniform: load them through the scalar unit so that
  // waiting for one never waits for the K/V vector loads in flight.
  const int nf = sload(a.n_full + qt), np = sload(a.n_part + qt), ntot = nf + np;
  const int32_t *frow = a.full_idx + (int64_t)qt * a.n_ktiles;
  const int32_t *prow = a.part_idx + (int64_t)qt * a.n_ktiles;
  auto tile_of = [&](int i) { return i < nf ? sload(frow + i) : sload(prow + i - nf); };

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = f32x16{};
  float m_run = -__builtin_inff();  // running max, in units of log2
  float l_run = 0.f;               // this lane's partial sum (its half of the keys)
  const float sl2 = a.scale_log2;
  const int krow = key_of_row(col);

  // Two register stagings for the K/V tiles in flight (each tile is loaded two
  // iterations ahead of its use) and two LDS stages. Iteration `it` writes LDS
  // stage it % 2; the last reader of that stage was iteration it - 2, and every
  // wave has passed iteration it - 1's barrier since, so one barrier per tile
  // suffices. The stagings are separate named arrays (not one array indexed by
  // the iteration) so they stay in registers.
  u32x4 kA[KPT], kB[KPT];
  uint32_t vA[VPT][8], vB[VPT][8];
  if (ntot > 0) load_tile<D, NT>(kA, vA, K, V, tile_of(0), tid);
  if (ntot > 1) load_tile<D, NT>(kB, vB, K, V, tile_of(1), tid);

  auto step = [&](auto &kst, auto &vst, const int it) __attribute__((always_inline)) {
      const int stage = it & 1;
      const int kt = tile_of(it);
      __bf16 *Ks = lds + stage * STAGE;
      __bf16 *Vs = Ks + BN * KS;
      store_tile<D, NT>(kst, vst, Ks, Vs, tid);
      __syncthreads();
      if (it + 2 < ntot) load_tile<D, NT>(kst, vst, K, V, tile_of(it + 2), tid);

      // S^T for the two 32-key blocks: all K operand reads issued first, then the
      // MFMAs with the two independent accumulators interleaved.
      bf16x8 kop[2][NCH];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const __bf16 *kr = Ks + (kb * 32 + krow) * KS + half * (D / 2);
#pragma unroll
        for (int c = 0; c < NCH; ++c) kop[kb][c] = *reinterpret_cast<const bf16x8 *>(kr + 8 * c);
      }
      f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
          s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kop[kb][c], qop[c], s[kb], 0, 0, 0);

      // V operand reads do not depend on the softmax: issue them now so their
      // latency hides behind it.
      bf16x8 vop[NDB][4];
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const __bf16 *vr = Vs + (db * 32 + col) * VS + 8 * half;
#pragma unroll
        for (int t = 0; t < 4; ++t) vop[db][t] = *reinterpret_cast<const bf16x8 *>(vr + 16 * t);
      }

      if (it >= nf) {  // partial tile: element mask
        const int kbase = kt * BN + 8 * half;  // first key of this lane's runs (multiple of 8)
        if (one_d) {
          // allowed iff lo <= key <= hi, as one unsigned compare
          const int base = kbase - lo;
          const uint32_t span = (uint32_t)(hi - lo);
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              const bool ok = (uint32_t)(base + kb * 32 + 16 * (v >> 3) + (v & 7)) <= span;
              s[kb][v] = ok ? s[kb][v] : -__builtin_inff();
            }
        } else if (row_runs) {
          // W % 8 == 0: each aligned run of 8 keys lies in one grid row, so one
          // division per run gives the row and the first column
          const uint32_t rspan = (uint32_t)(rhi - rlo), cspan = (uint32_t)(chi - clo);
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int g = 0; g < 2; ++g) {
              const int k0 = kbase + kb * 32 + 16 * g;
              const int r = (int)fdiv((uint32_t)k0, P.wdiv);
              const int c0 = k0 - r * P.W - clo;
              const bool row_ok = (uint32_t)(r - rlo) <= rspan;
#pragma unroll
              for (int t = 0; t < 8; ++t) {
                const bool ok = row_ok & ((uint32_t)(c0 + t) <= cspan);
                s[kb][8 * g + t] = ok ? s[kb][8 * g + t] : -__builtin_inff();
              }
            }
        } else {
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              const int kpos = kbase + kb * 32 + 16 * (v >> 3) + (v & 7);
              const int r = (int)fdiv((uint32_t)kpos, P.wdiv), c = kpos - r * P.W;
              const bool ok = (r >= rlo) & (r <= rhi) & (c >= clo) & (c <= chi);
              s[kb][v] = ok ? s[kb][v] : -__builtin_inff();
            }
        }
      }

      // Online softmax in the log2 domain with a lazily moved reference: the
      // exponent reference m_run only moves when a row's tile max exceeds it by
      // more than kRescaleSlack, so the O / l rescale is rare. Weights stay
      // <= 2^kRescaleSlack; the result is unchanged because O and l always share
      // the same reference.
      float mx = s[0][0];
#pragma unroll
      for (int v = 1; v < 16; ++v) mx = fmaxf(mx, s[0][v]);
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[1][v]);
      mx = xhalf_max(mx);
      const float mt = mx * sl2;
      const bool grow = mt > m_run + kRescaleSlack;
      if (__ballot(grow)) {
        const float m_new = grow ? mt : m_run;
        // 1 where unchanged; a row with no allowed key yet has nothing to rescale
        const float alpha = m_new == -__builtin_inff() ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < NDB; ++db) oacc[db] *= alpha;
        m_run = m_new;
      }
      const float m_use = m_run == -__builtin_inff() ? 0.f : m_run;
      // Row sums in fp32 from the unrounded weights (the log-sum-exp needs them to
      // better than bf16 precision); P goes to the PV product rounded to bf16.
      bf16x8 pop[4];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float pv = __builtin_amdgcn_exp2f(s[kb][v] * sl2 - m_use);
          l_run += pv;
          pop[kb * 2 + (v >> 3)][v & 7] = (__bf16)pv;
        }
      }

      // O^T += V^T P^T over four 16-key steps, d blocks interleaved.
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int db = 0; db < NDB; ++db)
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vop[db][t], pop[t], oacc[db], 0, 0, 0);
  };

  for (int it = 0; it < ntot; it += 2) {
    step(kA, vA, it);
    if (it + 1 < ntot) step(kB, vB, it + 1);
  }

  // Epilogue: normalise, stage O through LDS, write rows coalesced.
  const float l_tot = xhalf_sum(l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  __syncthreads();  // every wave is done reading K/V from LDS
  constexpr int OS = D + 8;
  __bf16 *Os = lds + wave * 32 * OS;
#pragma unroll
  for (int db = 0; db < NDB; ++db) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bf16x4 o4;
#pragma unroll
      for (int b = 0; b < 4; ++b) o4[b] = (__bf16)(oacc[db][4 * g + b] * inv);
      *reinterpret_cast<bf16x4 *>(Os + col * OS + db * 32 + 8 * g + 4 * half) = o4;
    }
  }
  __syncthreads();
  __bf16 *O = static_cast<__bf16 *>(a.out) + slice + (int64_t)(q0 + wave * 32) * D;
  constexpr int CPR = D / 8;  // 16-byte chunks per row
#pragma unroll
  for (int i = lane; i < 32 * CPR; i += 64) {
    const int r = i / CPR, c = i % CPR;
    *reinterpret_cast<uint4 *>(O + r * D + c * 8) =
        *reinterpret_cast<const uint4 *>(Os + r * OS + c * 8);
  }
  if (a.lse && half == 0) {
    const float ln2 = 0.69314718055994530942f;
    a.lse[(int64_t)bh * a.N + qpos] =
        l_tot > 0.f ? (m_run + __builtin_amdgcn_logf(l_tot)) * ln2 : -__builtin_inff();
  }
}

template <int D, int NW>
hipError_t launch(const AttnArgs &a, hipStream_t s) {
  const int64_t blocks = (int64_t)a.BH * a.n_qtiles;
  hipLaunchKernelGGL((attn_fwd_bf16<D, NW>), dim3((uint32_t)blocks), dim3(64 * NW), 0, s, a);
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
