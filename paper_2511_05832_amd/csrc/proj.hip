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
#include "hla_internal.h"

namespace hla {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kWaves = 4;
constexpr int kTokens = 32 * kWaves;
constexpr int kXcds = 8;

struct ProjArgs {
  const __bf16 *in;   // x [T, K] (QKV) or o [B, heads, N, d] (out)
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
        src = p.in + (int64_t)tt * p.K + k;
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
        dst = p.out0 + (int64_t)tt * p.F + feat;
      }
      *reinterpret_cast<bf16x4 *>(dst) = o4;
    }
  }
  }
}

template <int MODE>
hipError_t launch_fb(ProjArgs p, hipStream_t s) {
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

hipError_t launch_qkv_proj(const void *x, const void *w, void *q, void *k, void *v,
                           int64_t B, int64_t N, int64_t heads, int64_t d,
                           hipStream_t s) {
  ProjArgs p;
  p.in = static_cast<const __bf16 *>(x);
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

hipError_t launch_out_proj(const void *o, const void *w, void *y, int64_t B, int64_t N,
                           int64_t heads, int64_t d, int64_t c_out, hipStream_t s) {
  ProjArgs p;
  p.in = static_cast<const __bf16 *>(o);
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
