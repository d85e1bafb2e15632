// Per-row statistics for the attention backward pass.
//
// The softmax gradient of a row needs sum_j P_ij dP_ij, which equals
// delta_i = <dout_i, out_i> because out_i = sum_j P_ij v_j and dP_ij =
// <dout_i, v_j>. Each row's pair (lse_i * log2 e, delta_i) is written side by side
// so that the gradient kernels fetch both with one 8-byte access (and one
// 16-byte copy covers two rows). A row with lse = -inf (no allowed key) gets
// +inf in place of lse * log2 e, which makes every recomputed weight
// exp2(s - (+inf)) = 0 without a special case in the gradient kernels.
//
// Bound by HBM: reads out and dout once (2 * rows * d * sizeof(T) bytes) plus the
// lse, writes 8 bytes per row. LPR lanes share a row, one 16-byte load of each
// tensor per lane, reduced with cross-lane shuffles.
#include "hla_internal.h"

namespace hla {
namespace {

constexpr int kThreads = 256;

template <typename T>
__device__ __forceinline__ float to_f32(T x) {
  return (float)x;
}

template <typename T, int D>
__global__ void __launch_bounds__(kThreads)
    bwd_stats(const T *__restrict__ out, const T *__restrict__ dout,
              const float *__restrict__ lse, float *__restrict__ stats, int64_t rows) {
  constexpr int EPL = 16 / (int)sizeof(T);  // elements per lane
  constexpr int LPR = D / EPL;              // lanes per row (power of two, <= 16)
  constexpr int RPB = kThreads / LPR;       // rows per block
  typedef T vec_t __attribute__((ext_vector_type(EPL)));
  const int64_t row = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR;
  const int sub = threadIdx.x % LPR;
  float acc = 0.f;
  if (row < rows) {
    const vec_t o = *reinterpret_cast<const vec_t *>(out + row * D + sub * EPL);
    const vec_t g = *reinterpret_cast<const vec_t *>(dout + row * D + sub * EPL);
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc = __builtin_fmaf(to_f32(o[e]), to_f32(g[e]), acc);
  }
#pragma unroll
  for (int o = LPR / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if (row < rows && sub == 0) {
    const float l = lse[row];
    const float l2 = l == -__builtin_inff() ? __builtin_inff() : l * 1.4426950408889634f;
    *reinterpret_cast<float2 *>(stats + 2 * row) = make_float2(l2, acc);
  }
}

template <typename T, int D>
hipError_t launch(const AttnBwdArgs &a, hipStream_t s) {
  constexpr int LPR = D / (16 / (int)sizeof(T));
  const int64_t rows = (int64_t)a.BH * a.N;
  const int64_t rpb = kThreads / LPR;
  const int64_t blocks = (rows + rpb - 1) / rpb;
  hipLaunchKernelGGL((bwd_stats<T, D>), dim3((uint32_t)blocks), dim3(kThreads), 0, s,
                     static_cast<const T *>(a.out), static_cast<const T *>(a.dout), a.lse,
                     a.stats, rows);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd_stats(const AttnBwdArgs &a, int d, bool bf16, hipStream_t s) {
  if (bf16) return d == 64 ? launch<__bf16, 64>(a, s) : launch<__bf16, 32>(a, s);
  return d == 64 ? launch<float, 64>(a, s) : launch<float, 32>(a, s);
}

}  // namespace hla
