// Gather into / scatter out of Hilbert order: the paper's "reshape" step
// (Sec. 4.2, input processing; Tables 8 and 10, Reshape column).
//
//   gather:  dst[bh, i, :]        = src[bh, order[i], :]
//   scatter: dst[bh, order[i], :] = src[bh, i, :]
//
// Pure data movement, bound by HBM bandwidth: every row is read once and
// written once (2 * B*heads*N*row_bytes bytes + 4N bytes of index). A row is
// row_bytes contiguous bytes (128 B for d = 64 in bf16), so one index lookup
// moves a whole row. Each thread moves UNROLL vector chunks of VEC bytes, all
// loads issued before the stores, so a wave keeps UNROLL * 64 * VEC bytes in
// flight. The sequential side (dst for gather, src for scatter) is accessed
// fully coalesced; the permuted side touches whole rows, so every 64-byte
// segment it touches is used in full.
#include "hla_internal.h"

namespace hla {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

template <int VEC>
struct Vec;
template <>
struct Vec<16> {
  using T = uint4;
};
template <>
struct Vec<8> {
  using T = uint2;
};
template <>
struct Vec<4> {
  using T = uint32_t;
};

// grid: x = ceil(N * chunks_per_row / (kThreads * kUnroll)), y = B*heads slices
template <int VEC, bool SCATTER>
__global__ void __launch_bounds__(kThreads)
    permute_rows(const char *__restrict__ src, char *__restrict__ dst,
                 const int32_t *__restrict__ order, uint32_t N, uint32_t cpr,
                 FastDiv cpr_div, uint64_t slice_bytes) {
  using T = typename Vec<VEC>::T;
  const uint32_t total = N * cpr;
  const uint64_t base = (uint64_t)blockIdx.y * slice_bytes;
  const T *s = reinterpret_cast<const T *>(src + base);
  T *o = reinterpret_cast<T *>(dst + base);
  const uint32_t first = blockIdx.x * (kThreads * kUnroll) + threadIdx.x;
  T buf[kUnroll];
  uint32_t dst_idx[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const uint32_t g = first + u * kThreads;
    dst_idx[u] = 0xffffffffu;
    if (g < total) {
      const uint32_t i = fdiv(g, cpr_div);
      const uint32_t c = g - i * cpr;
      const uint32_t p = (uint32_t)__ldg(order + i);
      if (SCATTER) {
        buf[u] = s[g];
        dst_idx[u] = p * cpr + c;
      } else {
        buf[u] = s[p * cpr + c];
        dst_idx[u] = g;
      }
    }
  }
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    if (dst_idx[u] != 0xffffffffu) o[dst_idx[u]] = buf[u];
  }
}

template <int VEC>
hipError_t launch_vec(const void *src, void *dst, const int32_t *order, int64_t BH,
                      int64_t N, int64_t row_bytes, bool scatter, hipStream_t s) {
  const uint32_t cpr = (uint32_t)(row_bytes / VEC);
  const uint64_t total = (uint64_t)N * cpr;
  const uint32_t blocks = (uint32_t)((total + kThreads * kUnroll - 1) / (kThreads * kUnroll));
  const uint64_t slice = (uint64_t)N * (uint64_t)row_bytes;
  const FastDiv fd = make_fastdiv(cpr);
  // grid.y is limited to 65535 slices per launch; loop over larger batches
  for (int64_t b0 = 0; b0 < BH; b0 += 65535) {
    const uint32_t nb = (uint32_t)((BH - b0) < 65535 ? (BH - b0) : 65535);
    const char *sp = static_cast<const char *>(src) + (uint64_t)b0 * slice;
    char *dp = static_cast<char *>(dst) + (uint64_t)b0 * slice;
    if (scatter)
      hipLaunchKernelGGL((permute_rows<VEC, true>), dim3(blocks, nb), dim3(kThreads), 0, s,
                         sp, dp, order, (uint32_t)N, cpr, fd, slice);
    else
      hipLaunchKernelGGL((permute_rows<VEC, false>), dim3(blocks, nb), dim3(kThreads), 0, s,
                         sp, dp, order, (uint32_t)N, cpr, fd, slice);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace

hipError_t launch_permute(const void *src, void *dst, const int32_t *order,
                          int64_t BH, int64_t N, int64_t row_bytes, bool scatter,
                          hipStream_t s) {
  if (row_bytes % 16 == 0) return launch_vec<16>(src, dst, order, BH, N, row_bytes, scatter, s);
  if (row_bytes % 8 == 0) return launch_vec<8>(src, dst, order, BH, N, row_bytes, scatter, s);
  return launch_vec<4>(src, dst, order, BH, N, row_bytes, scatter, s);
}

}  // namespace hla
