// Block-sparse attention forward in fp32 throughout (fp32 I/O, fp32 products).
//
// Same algorithm as the bf16 kernel (Sec. 3.1; Eq. 1: only the listed key
// tiles are visited, full tiles unmasked, partial tiles masked, online
// softmax), written for exact fp32 arithmetic: gfx950 has no reduced-precision
// fp32 matrix mode, and fp32 vector FMA runs at the same 157 TFLOP/s as fp32
// MFMA, so the products are plain FMAs. Four lanes share a query row, each
// owning a quarter of d: a score is four partial dot products summed across the
// four lanes (two exchanges), and each lane accumulates its quarter of the
// output row. (One lane per row left the small fp32 workload - a thousand rows
// - with one wave per CU on 16 CUs, each running a 4096-FMA dependent chain per
// key tile.) K and V tiles are staged in LDS; at a key, the lanes of a wave read
// four distinct 16-byte pieces. MODE ATTN_GATHER: the tensors are stored in
// grid order and sequence position i lives in row a.order[i] (reordering fused
// into the loads and stores). MODE ATTN_RPB: every score gets the global
// relative position bias of the grid cells order[i], order[j] (see the bf16
// kernel).
#include "attn_common.h"

namespace hla {
namespace {

constexpr int BN = 64;
constexpr int CH = 16;   // keys per online-softmax step
constexpr int LPR = 4;   // lanes per query row

template <int D, int BM, int MODE>
__global__ void __launch_bounds__(BM * LPR) attn_fwd_f32(AttnArgs a) {
  constexpr bool GATHER = MODE == ATTN_GATHER;
  constexpr bool RPB = MODE == ATTN_RPB;
  constexpr int NT = BM * LPR;
  constexpr int DL = D / LPR;  // dims per lane
  static_assert(DL % 4 == 0, "a lane's dims are whole float4s");
  __shared__ __attribute__((aligned(16))) float Ks[BN * D];
  __shared__ __attribute__((aligned(16))) float Vs[BN * D];

  const int tid = threadIdx.x;
  const int row = tid / LPR, i0 = (tid % LPR) * DL;  // this lane's row and first dim
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = logical / a.n_qtiles;
  const int qt = logical - bh * a.n_qtiles;
  const int qpos = qt * BM + row;
  const int64_t slice = (int64_t)bh * a.N * D;
  const float *Q = static_cast<const float *>(a.q) + slice;
  const float *K = static_cast<const float *>(a.k) + slice;
  const float *V = static_cast<const float *>(a.v) + slice;

  // A query row past the end of the sequence (ragged last query tile) reads row
  // N - 1 and stores nothing; key rows past it read row N - 1 and are masked
  // (such a tile is always partial and every allowed region ends at N - 1).
  const bool live = qpos < a.N;
  const int qc = min(qpos, a.N - 1);
  const int64_t qrow = GATHER ? (int64_t)a.order[qc] : (int64_t)qc;
  float q[DL], acc[DL];
#pragma unroll
  for (int i = 0; i < DL; i += 4) {
    const float4 t = *reinterpret_cast<const float4 *>(Q + qrow * D + i0 + i);
    q[i] = t.x; q[i + 1] = t.y; q[i + 2] = t.z; q[i + 3] = t.w;
  }
#pragma unroll
  for (int i = 0; i < DL; ++i) acc[i] = 0.f;

  const PatternArgs &P = a.pat;
  const Region R = region_of<true>(P, qpos);

  const int nf = a.n_full[qt], np = a.n_part[qt], ntot = nf + np;
  const int32_t *frow = a.full_idx + (int64_t)qt * a.n_ktiles;
  const int32_t *prow = a.part_idx + (int64_t)qt * a.n_ktiles;
  // scores are multiplied by smul to reach log2 units (RPB: already scaled)
  const float sl2 = RPB ? 1.44269504088896340736f : a.scale_log2;
  float m_run = -__builtin_inff(), l_run = 0.f;
  int32_t rpb_base = 0;
  const float *rpb_h = nullptr;
  if constexpr (RPB) {
    const int32_t g = a.order[qc];
    rpb_base = (P.H - 1) * (2 * P.W - 1) + (P.W - 1) + g + (P.W - 1) * (int32_t)fdiv((uint32_t)g, P.wdiv);
    rpb_h = a.rpb + (int64_t)(bh % a.heads) * (2 * P.H - 1) * (2 * P.W - 1);
  }

  for (int it = 0; it < ntot; ++it) {
    const bool masked = it >= nf;
    const int kt = masked ? prow[it - nf] : frow[it];
    __syncthreads();
    for (int i = tid; i < BN * D / 4; i += NT) {
      const int r = i / (D / 4), c4 = i % (D / 4);
      const int pos = min(kt * BN + r, a.N - 1);
      const int64_t krow = GATHER ? (int64_t)a.order[pos] : (int64_t)pos;
      reinterpret_cast<float4 *>(Ks)[i] = reinterpret_cast<const float4 *>(K + krow * D)[c4];
      reinterpret_cast<float4 *>(Vs)[i] = reinterpret_cast<const float4 *>(V + krow * D)[c4];
    }
    __syncthreads();
    for (int j0 = 0; j0 < BN; j0 += CH) {
      float s[CH];
#pragma unroll
      for (int j = 0; j < CH; ++j) {
        float dot = 0.f;
#pragma unroll
        for (int i = 0; i < DL; i += 4) {
          const float4 k4 = *reinterpret_cast<const float4 *>(Ks + (j0 + j) * D + i0 + i);
          dot = __builtin_fmaf(q[i], k4.x, dot);
          dot = __builtin_fmaf(q[i + 1], k4.y, dot);
          dot = __builtin_fmaf(q[i + 2], k4.z, dot);
          dot = __builtin_fmaf(q[i + 3], k4.w, dot);
        }
        // the row's four partial sums, in the same order in all four lanes
        // ((l0 + l1) + (l2 + l3)), so they agree on the score bit for bit
        dot += __shfl_xor(dot, 1);
        dot += __shfl_xor(dot, 2);
        s[j] = dot;
        if constexpr (RPB) {
          const int32_t gk = a.order[min(kt * BN + j0 + j, a.N - 1)];
          const int32_t koff = gk + (P.W - 1) * (int32_t)fdiv((uint32_t)gk, P.wdiv);
          s[j] = __builtin_fmaf(dot, a.scale, rpb_h[rpb_base - koff]);
        }
      }
      if (masked) {
#pragma unroll
        for (int j = 0; j < CH; ++j)
          if (!region_has(R, P, kt * BN + j0 + j)) s[j] = -__builtin_inff();
      }
      float mx = s[0];
#pragma unroll
      for (int j = 1; j < CH; ++j) mx = fmaxf(mx, s[j]);
      const float m_new = fmaxf(m_run, mx * sl2);
      const float m_use = m_new == -__builtin_inff() ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int i = 0; i < DL; ++i) acc[i] *= alpha;
#pragma unroll
      for (int j = 0; j < CH; ++j) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[j], sl2, -m_use));
        l_run += p;
#pragma unroll
        for (int i = 0; i < DL; i += 4) {
          const float4 v4 = *reinterpret_cast<const float4 *>(Vs + (j0 + j) * D + i0 + i);
          acc[i] = __builtin_fmaf(p, v4.x, acc[i]);
          acc[i + 1] = __builtin_fmaf(p, v4.y, acc[i + 1]);
          acc[i + 2] = __builtin_fmaf(p, v4.z, acc[i + 2]);
          acc[i + 3] = __builtin_fmaf(p, v4.w, acc[i + 3]);
        }
      }
    }
  }

  if (!live) return;
  const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
  float *O = static_cast<float *>(a.out) + slice + qrow * D + i0;
#pragma unroll
  for (int i = 0; i < DL; i += 4)
    *reinterpret_cast<float4 *>(O + i) =
        make_float4(acc[i] * inv, acc[i + 1] * inv, acc[i + 2] * inv, acc[i + 3] * inv);
  if (a.lse && i0 == 0) {
    const float ln2 = 0.69314718055994530942f;
    a.lse[(int64_t)bh * a.N + qrow] =
        l_run > 0.f ? (m_run + __builtin_amdgcn_logf(l_run)) * ln2 : -__builtin_inff();
  }
}

template <int D, int BM>
hipError_t launch(const AttnArgs &a, hipStream_t s) {
  const int64_t blocks = (int64_t)a.BH * a.n_qtiles;
  if (a.mode == ATTN_GATHER)
    hipLaunchKernelGGL((attn_fwd_f32<D, BM, ATTN_GATHER>), dim3((uint32_t)blocks), dim3(BM * LPR), 0, s, a);
  else if (a.mode == ATTN_RPB)
    hipLaunchKernelGGL((attn_fwd_f32<D, BM, ATTN_RPB>), dim3((uint32_t)blocks), dim3(BM * LPR), 0, s, a);
  else
    hipLaunchKernelGGL((attn_fwd_f32<D, BM, ATTN_PLAIN>), dim3((uint32_t)blocks), dim3(BM * LPR), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_f32(const AttnArgs &a, int d, int tile_m, int tile_n,
                           hipStream_t s) {
  if (tile_n != BN) return hipErrorInvalidValue;
  if (d == 32 && tile_m == 64) return launch<32, 64>(a, s);
  if (d == 32 && tile_m == 128) return launch<32, 128>(a, s);
  if (d == 64 && tile_m == 64) return launch<64, 64>(a, s);
  if (d == 64 && tile_m == 128) return launch<64, 128>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace hla
