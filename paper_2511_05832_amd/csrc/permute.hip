// Gather into / scatter out of Hilbert order: the paper's "reshape" step
// (Sec. 4.2, input processing; Tables 8 and 10, Reshape column).
//
//   gather:  dst[bh, i, :]        = src[bh, order[i], :]
//   scatter: dst[bh, order[i], :] = src[bh, i, :]
//
// Pure data movement, bound by HBM bandwidth: every row is read once and
// written once (2 * B*heads*N*row_bytes bytes + 4N bytes of index). A row is
// row_bytes contiguous bytes (128 B for d = 64 in bf16), so one index lookup
// moves a whole row. The sequential side (dst for gather, src for scatter) is
// accessed fully coalesced; the permuted side touches whole rows, so every
// segment it touches is used in full. A random order costs no more than the
// identity here: the limit is the kernel's issue structure, not row locality.
#include "hla_internal.h"

namespace hla {
namespace {

// One 16-byte chunk per thread per iteration measured fastest on MI355X (5.0-5.3
// TB/s at 64 MiB per tensor, against 5.1 TB/s for hipMemcpy device to device);
// more chunks per thread, 512-thread blocks and non-temporal accesses were not.
constexpr int kThreads = 256;
constexpr int kUnroll = 1;

template <int VEC>
struct Vec;
template <>
struct Vec<16> {
  using T = uint32_t __attribute__((ext_vector_type(4)));
};
template <>
struct Vec<8> {
  using T = uint32_t __attribute__((ext_vector_type(2)));
};
template <>
struct Vec<4> {
  using T = uint32_t;
};

// Persistent grid-stride kernel over "blocks" of kThreads * kUnroll chunks; a
// block lies inside one (b, head) slice. The permuted side needs order[i] before
// its data load can issue, so the indices of the next block are loaded while the
// current block's data loads are in flight: the index latency overlaps the data
// latency instead of adding to it.
template <int VEC, bool SCATTER>
__global__ void __launch_bounds__(kThreads)
    permute_rows(const char *__restrict__ src, char *__restrict__ dst,
                 const int32_t *__restrict__ order, uint32_t N, uint32_t cpr,
                 FastDiv cpr_div, uint64_t slice_bytes, uint32_t blocks_per_slice,
                 uint32_t total_blocks) {
  using T = typename Vec<VEC>::T;
  constexpr uint32_t kChunks = kThreads * kUnroll;
  const uint32_t total = N * cpr;

  uint32_t blk = blockIdx.x;
  if (blk >= total_blocks) return;
  // Chunk g of a slice is row g / cpr, column g % cpr. Whole blocks take an
  // unguarded path so all kUnroll loads issue back to back; only the ragged last
  // block of a slice checks bounds per chunk.
  uint32_t pidx[kUnroll];
  auto load_idx = [&](uint32_t b) {
    const uint32_t first = (b % blocks_per_slice) * kChunks + threadIdx.x;
    if (first - threadIdx.x + kChunks <= total) {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
        pidx[u] = (uint32_t)__ldg(order + fdiv(first + u * kThreads, cpr_div));
    } else {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const uint32_t g = first + u * kThreads;
        pidx[u] = (uint32_t)__ldg(order + fdiv(g < total ? g : total - 1, cpr_div));
      }
    }
  };
  load_idx(blk);
  for (; blk < total_blocks; blk += gridDim.x) {
    const uint32_t slice = blk / blocks_per_slice;
    const uint32_t first = (blk - slice * blocks_per_slice) * kChunks + threadIdx.x;
    const T *s = reinterpret_cast<const T *>(src + (uint64_t)slice * slice_bytes);
    T *o = reinterpret_cast<T *>(dst + (uint64_t)slice * slice_bytes);
    const bool whole = first - threadIdx.x + kChunks <= total;
    T buf[kUnroll];
    uint32_t sidx[kUnroll], didx[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const uint32_t g = whole ? first + u * kThreads : min(first + u * kThreads, total - 1);
      const uint32_t i = fdiv(g, cpr_div);
      const uint32_t c = g - i * cpr;
      sidx[u] = SCATTER ? g : pidx[u] * cpr + c;
      didx[u] = SCATTER ? pidx[u] * cpr + c : g;
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) buf[u] = s[sidx[u]];
    const uint32_t nxt = blk + gridDim.x;
    if (nxt < total_blocks) load_idx(nxt);
    if (whole) {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) o[didx[u]] = buf[u];
    } else {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
        if (first + u * kThreads < total) o[didx[u]] = buf[u];
    }
  }
}

int resident_blocks() {
  static int n = 0;
  if (!n) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
    n = cus * (2048 / kThreads);  // 8 waves per SIMD
  }
  return n;
}

template <int VEC>
hipError_t launch_vec(const void *src, void *dst, const int32_t *order, int64_t BH,
                      int64_t N, int64_t row_bytes, bool scatter, hipStream_t s) {
  const uint32_t cpr = (uint32_t)(row_bytes / VEC);
  const uint64_t total = (uint64_t)N * cpr;
  const uint32_t per_slice = (uint32_t)((total + kThreads * kUnroll - 1) / (kThreads * kUnroll));
  const uint64_t slice = (uint64_t)N * (uint64_t)row_bytes;
  const FastDiv fd = make_fastdiv(cpr);
  // launch over batches of slices so that the block count fits in 32 bits
  const int64_t max_slices = (int64_t)(0x7fffffffu / per_slice);
  for (int64_t b0 = 0; b0 < BH; b0 += max_slices) {
    const int64_t nb = (BH - b0) < max_slices ? (BH - b0) : max_slices;
    const uint32_t nblocks = (uint32_t)(nb * per_slice);
    const uint32_t grid = nblocks < (uint32_t)resident_blocks() ? nblocks : (uint32_t)resident_blocks();
    const char *sp = static_cast<const char *>(src) + (uint64_t)b0 * slice;
    char *dp = static_cast<char *>(dst) + (uint64_t)b0 * slice;
    if (scatter)
      hipLaunchKernelGGL((permute_rows<VEC, true>), dim3(grid), dim3(kThreads), 0, s, sp, dp,
                         order, (uint32_t)N, cpr, fd, slice, per_slice, nblocks);
    else
      hipLaunchKernelGGL((permute_rows<VEC, false>), dim3(grid), dim3(kThreads), 0, s, sp, dp,
                         order, (uint32_t)N, cpr, fd, slice, per_slice, nblocks);
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
