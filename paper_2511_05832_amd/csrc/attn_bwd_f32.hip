// Block-sparse attention backward in fp32 throughout (fp32 I/O, fp32 products).
//
// Same computation and tile walk as the bf16 backward (gradients of the forward
// over the listed tiles only; P and dP recomputed from the forward's lse and the
// row statistics; no atomics), in exact fp32 with plain FMAs: as in the fp32
// forward, gfx950's fp32 vector rate equals its fp32 matrix rate. A row of d
// values is split over TPR = d/32 threads of 32 values each, whose partial dot
// products are combined with one cross-lane exchange.
//
//   dq kernel    one thread group per query row; K and V tiles of the row list
//                staged in LDS and read as broadcasts; it also computes the row's
//                statistics (lse * log2 e, -delta; delta = <dout, out>) and stores them.
//   dkdv kernel  one thread group per key row; query, dout and stats tiles of
//                the column list staged in LDS, QC query rows at a time.
#include "attn_common.h"

namespace hla {
namespace {

constexpr int BN = 64;
constexpr int E = 32;  // values of a row per thread

template <int TPR>
__device__ __forceinline__ float row_sum(float x) {
  if (TPR == 2) x += __shfl_xor(x, 1);
  return x;
}

template <int D, int BM>
__global__ void __launch_bounds__(BM * (D / E)) attn_bwd_dq_f32(AttnBwdArgs a) {
  constexpr int TPR = D / E;
  constexpr int NT = BM * TPR;
  __shared__ __attribute__((aligned(16))) float Ks[BN * D];
  __shared__ __attribute__((aligned(16))) float Vs[BN * D];

  const int tid = threadIdx.x, part = tid % TPR;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = logical / a.n_qtiles;
  const int qt = logical - bh * a.n_qtiles;
  const int qpos = qt * BM + tid / TPR;
  const int64_t slice = (int64_t)bh * a.N * D;
  const float *Q = static_cast<const float *>(a.q) + slice;
  const float *K = static_cast<const float *>(a.k) + slice;
  const float *V = static_cast<const float *>(a.v) + slice;
  const float *G = static_cast<const float *>(a.dout) + slice;

  // A query row past the end of the sequence (ragged last query tile) reads row
  // N - 1 and stores nothing; key rows past it read row N - 1 and are masked.
  // With an order (fused reordering) sequence position i is stored in row order[i].
  auto row_of = [&](int i) -> int64_t { return a.order ? (int64_t)a.order[i] : (int64_t)i; };
  const int64_t qrow = row_of(min(qpos, a.N - 1));
  float q[E], g[E], acc[E];
#pragma unroll
  for (int i = 0; i < E; ++i) {
    q[i] = Q[qrow * D + part * E + i];
    g[i] = G[qrow * D + part * E + i];
    acc[i] = 0.f;
  }
  // This query's row statistics, computed here and stored for the dk/dv kernel:
  // (lse * log2 e, +inf for a row with no allowed key; delta = <dout, out>).
  const float *O = static_cast<const float *>(a.out) + slice;
  float dpart = 0.f;
#pragma unroll
  for (int i = 0; i < E; ++i) dpart = __builtin_fmaf(O[qrow * D + part * E + i], g[i], dpart);
  const float lraw = a.lse[(int64_t)bh * a.N + qrow];
  const float2 rs = make_float2(lraw == -__builtin_inff() ? __builtin_inff() : lraw * 1.4426950408889634f,
                                row_sum<TPR>(dpart));
  // stored as (lse log2e, -delta), the workspace's layout
  if (part == 0 && qpos < a.N)
    *reinterpret_cast<float2 *>(a.stats + 2 * ((int64_t)bh * a.N + qrow)) = make_float2(rs.x, -rs.y);
  const PatternArgs &P = a.pat;
  const Region R = region_of<true>(P, qpos);
  const float sl2 = a.scale_log2;

  const int nf = a.n_full[qt], np = a.n_part[qt], ntot = nf + np;
  const int32_t *frow = a.full_idx + (int64_t)qt * a.n_ktiles;
  const int32_t *prow = a.part_idx + (int64_t)qt * a.n_ktiles;
  for (int it = 0; it < ntot; ++it) {
    const bool masked = it >= nf;
    const int kt = masked ? prow[it - nf] : frow[it];
    __syncthreads();
    for (int i = tid; i < BN * D / 4; i += NT) {
      const int64_t row = row_of(min(kt * BN + i / (D / 4), a.N - 1));
      reinterpret_cast<float4 *>(Ks)[i] = reinterpret_cast<const float4 *>(K + row * D)[i % (D / 4)];
      reinterpret_cast<float4 *>(Vs)[i] = reinterpret_cast<const float4 *>(V + row * D)[i % (D / 4)];
    }
    __syncthreads();
    for (int j = 0; j < BN; ++j) {
      const float *kr = Ks + j * D + part * E;
      const float *vr = Vs + j * D + part * E;
      float s = 0.f, dp = 0.f;
#pragma unroll
      for (int i = 0; i < E; ++i) {
        s = __builtin_fmaf(q[i], kr[i], s);
        dp = __builtin_fmaf(g[i], vr[i], dp);
      }
      s = row_sum<TPR>(s);
      dp = row_sum<TPR>(dp);
      const bool ok = !masked || region_has(R, P, kt * BN + j);
      const float p = ok ? __builtin_amdgcn_exp2f(__builtin_fmaf(s, sl2, -rs.x)) : 0.f;
      const float ds = p * (dp - rs.y);
#pragma unroll
      for (int i = 0; i < E; ++i) acc[i] = __builtin_fmaf(ds, kr[i], acc[i]);
    }
  }
  if (qpos >= a.N) return;
  float *dQ = static_cast<float *>(a.dq) + slice + qrow * D + part * E;
#pragma unroll
  for (int i = 0; i < E; i += 4)
    *reinterpret_cast<float4 *>(dQ + i) =
        make_float4(acc[i] * a.scale, acc[i + 1] * a.scale, acc[i + 2] * a.scale, acc[i + 3] * a.scale);
}

template <int D, int BMQ>
__global__ void __launch_bounds__(BN * (D / E)) attn_bwd_dkdv_f32(AttnBwdArgs a) {
  constexpr int TPR = D / E;
  constexpr int NT = BN * TPR;
  constexpr int QC = BMQ < 64 ? BMQ : 64;  // query rows staged at a time
  __shared__ __attribute__((aligned(16))) float Qs[QC * D];
  __shared__ __attribute__((aligned(16))) float Gs[QC * D];
  __shared__ __attribute__((aligned(16))) float Ss[2 * QC];

  const int tid = threadIdx.x, part = tid % TPR;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int bh = logical / a.n_ktiles;
  const int kt = logical - bh * a.n_ktiles;
  const int kpos = kt * BN + tid / TPR;
  const int64_t slice = (int64_t)bh * a.N * D;
  const float *Q = static_cast<const float *>(a.q) + slice;
  const float *K = static_cast<const float *>(a.k) + slice;
  const float *V = static_cast<const float *>(a.v) + slice;
  const float *G = static_cast<const float *>(a.dout) + slice;
  const float *S = a.stats + 2 * (int64_t)bh * a.N;

  // A key row past the end of the sequence (ragged last key tile) reads row
  // N - 1 and stores nothing; query rows past it read row N - 1 and are masked.
  // With an order (fused reordering) sequence position i is stored in row order[i].
  auto row_of = [&](int64_t i) -> int64_t { return a.order ? (int64_t)a.order[i] : i; };
  const int64_t krow = row_of(min(kpos, a.N - 1));
  float k[E], v[E], dk[E], dv[E];
#pragma unroll
  for (int i = 0; i < E; ++i) {
    k[i] = K[krow * D + part * E + i];
    v[i] = V[krow * D + part * E + i];
    dk[i] = 0.f;
    dv[i] = 0.f;
  }
  const PatternArgs &P = a.pat;
  const Region R = region_of<false>(P, kpos);
  const float sl2 = a.scale_log2;

  const int nf = a.n_full_t[kt], np = a.n_part_t[kt], ntot = nf + np;
  const int32_t *fcol = a.full_idx_t + (int64_t)kt * a.n_qtiles;
  const int32_t *pcol = a.part_idx_t + (int64_t)kt * a.n_qtiles;
  for (int it = 0; it < ntot; ++it) {
    const bool masked = it >= nf;
    const int qt = masked ? pcol[it - nf] : fcol[it];
    for (int c0 = 0; c0 < BMQ; c0 += QC) {
      const int64_t r0 = (int64_t)qt * BMQ + c0;
      __syncthreads();
      for (int i = tid; i < QC * D / 4; i += NT) {
        const int64_t row = row_of(min(r0 + i / (D / 4), (int64_t)a.N - 1));
        reinterpret_cast<float4 *>(Qs)[i] = reinterpret_cast<const float4 *>(Q + row * D)[i % (D / 4)];
        reinterpret_cast<float4 *>(Gs)[i] = reinterpret_cast<const float4 *>(G + row * D)[i % (D / 4)];
      }
      for (int i = tid; i < 2 * QC; i += NT) Ss[i] = S[2 * row_of(min(r0 + i / 2, (int64_t)a.N - 1)) + (i & 1)];
      __syncthreads();
      for (int j = 0; j < QC; ++j) {
        const float *qr = Qs + j * D + part * E;
        const float *gr = Gs + j * D + part * E;
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int i = 0; i < E; ++i) {
          s = __builtin_fmaf(qr[i], k[i], s);
          dp = __builtin_fmaf(gr[i], v[i], dp);
        }
        s = row_sum<TPR>(s);
        dp = row_sum<TPR>(dp);
        const bool ok = !masked || region_has(R, P, (int)r0 + j);
        const float p = ok ? __builtin_amdgcn_exp2f(__builtin_fmaf(s, sl2, -Ss[2 * j])) : 0.f;
        const float ds = p * (dp + Ss[2 * j + 1]);  // (the stats hold -delta)
#pragma unroll
        for (int i = 0; i < E; ++i) {
          dv[i] = __builtin_fmaf(p, gr[i], dv[i]);
          dk[i] = __builtin_fmaf(ds, qr[i], dk[i]);
        }
      }
    }
  }
  if (kpos >= a.N) return;
  float *dK = static_cast<float *>(a.dk) + slice + krow * D + part * E;
  float *dV = static_cast<float *>(a.dv) + slice + krow * D + part * E;
#pragma unroll
  for (int i = 0; i < E; i += 4) {
    *reinterpret_cast<float4 *>(dK + i) =
        make_float4(dk[i] * a.scale, dk[i + 1] * a.scale, dk[i + 2] * a.scale, dk[i + 3] * a.scale);
    *reinterpret_cast<float4 *>(dV + i) = make_float4(dv[i], dv[i + 1], dv[i + 2], dv[i + 3]);
  }
}

template <int D, int BM>
hipError_t launch_all(const AttnBwdArgs &a, hipStream_t s) {
  // the dq kernel also writes the row statistics the dk/dv kernel reads
  hipLaunchKernelGGL((attn_bwd_dq_f32<D, BM>), dim3((uint32_t)((int64_t)a.BH * a.n_qtiles)),
                     dim3(BM * (D / E)), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_bwd_dkdv_f32<D, BM>), dim3((uint32_t)((int64_t)a.BH * a.n_ktiles)),
                     dim3(BN * (D / E)), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bwd_f32(const AttnBwdArgs &a, int d, int tile_m, int tile_n,
                               hipStream_t s) {
  if (tile_n != BN) return hipErrorInvalidValue;
  if (d == 32 && tile_m == 64) return launch_all<32, 64>(a, s);
  if (d == 32 && tile_m == 128) return launch_all<32, 128>(a, s);
  if (d == 64 && tile_m == 64) return launch_all<64, 64>(a, s);
  if (d == 64 && tile_m == 128) return launch_all<64, 128>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace hla
