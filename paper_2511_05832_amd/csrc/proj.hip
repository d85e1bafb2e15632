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
        const int64_t yrow = p.order ? (int64_t)b * p.N + p.order[n] : (int64_t)tt;
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

template <int KC, int MODE>
hipError_t launch_rows(const ProjArgs &p, hipStream_t s) {
  const uint32_t gx = (uint32_t)((p.T + kTokens - 1) / kTokens);
  hipLaunchKernelGGL((proj_rows_kernel<KC, 3, MODE>), dim3(gx), dim3(64 * kWaves), 0, s, p);
  return hipGetLastError();
}

template <int MODE>
hipError_t launch_fb(ProjArgs p, hipStream_t s) {
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
