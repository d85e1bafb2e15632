// C-ABI entry points of libhla: argument validation on the host, then launch.
// Every check runs before the first HIP call, so a rejected call enqueues
// nothing and writes nothing.
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>

#include "hla_internal.h"

// Row statistics of the allocation-free backward (hla_attn_bwd_noalloc): two
// floats per (b, h, row), up to kScratchRows rows. Every device the library
// runs on holds its own copy for the life of the process. Host code never
// passes this name to a kernel (on the host it is only a stand-in for the
// symbol): it uses the address hipGetSymbolAddress returns for the current
// device, kept in g_scratch_ptr.
constexpr int64_t kScratchRows = 1LL << 20;
static __device__ __align__(256) float scratch[2 * kScratchRows];

namespace {

thread_local std::string g_last_error;

hla_status fail(hla_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

hla_status hip_status(hipError_t e, const char *what) {
  if (e == hipSuccess) return HLA_OK;
  return fail(HLA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }
int64_t dtype_size(hla_dtype dt) { return dt == HLA_F32 ? 4 : (dt == HLA_BF16 ? 2 : 0); }

constexpr int64_t kMaxI32 = 2147483647LL;

hla_status check_pattern(const hla_pattern_desc *p) {
  if (!p) return fail(HLA_ERR_INVALID_ARG, "pattern descriptor is NULL");
  if (p->H <= 0 || p->W <= 0) return fail(HLA_ERR_INVALID_ARG, "grid %dx%d must be positive", p->H, p->W);
  const int64_t N = (int64_t)p->H * p->W;
  if (N > (1LL << 30)) return fail(HLA_ERR_UNSUPPORTED, "N = %lld exceeds 2^30 tokens", (long long)N);
  if (p->p0 > (1 << 30) || p->p1 > (1 << 30))
    return fail(HLA_ERR_UNSUPPORTED, "pattern parameters above 2^30");
  switch (p->pattern) {
    case HLA_HILBERT_WINDOW:
      if (p->p0 < 1) return fail(HLA_ERR_INVALID_ARG, "window length p0 = %d must be >= 1", p->p0);
      break;
    case HLA_HILBERT_SLIDE:
      if (p->p0 < 0) return fail(HLA_ERR_INVALID_ARG, "half-width p0 = %d must be >= 0", p->p0);
      break;
    case HLA_HILBERT_NEIGHBORHOOD:
      if (p->p0 < 1 || p->p0 > N)
        return fail(HLA_ERR_INVALID_ARG, "neighbourhood length p0 = %d must be in [1, N]", p->p0);
      break;
    case HLA_HILBERT_SHIFTED_WINDOW:
      if (p->p0 < 1) return fail(HLA_ERR_INVALID_ARG, "window length p0 = %d must be >= 1", p->p0);
      if (p->p1 < 0 || p->p1 >= p->p0)
        return fail(HLA_ERR_INVALID_ARG, "shift p1 = %d must be in [0, window)", p->p1);
      break;
    case HLA_ROWMAJOR_WINDOW:
      if (p->p0 < 1 || p->p1 < 1)
        return fail(HLA_ERR_INVALID_ARG, "window %dx%d must be >= 1", p->p0, p->p1);
      break;
    case HLA_ROWMAJOR_SLIDE:
      if (p->p0 < 0 || p->p1 < 0)
        return fail(HLA_ERR_INVALID_ARG, "radii %d,%d must be >= 0", p->p0, p->p1);
      break;
    case HLA_ROWMAJOR_NEIGHBORHOOD:
      if (p->p0 < 1 || p->p1 < 1 || p->p0 > p->H || p->p1 > p->W)
        return fail(HLA_ERR_INVALID_ARG, "kernel %dx%d must be in [1,H]x[1,W]", p->p0, p->p1);
      break;
    default:
      return fail(HLA_ERR_INVALID_ARG, "unknown pattern %d", p->pattern);
  }
  return HLA_OK;
}

hla_status check_tiles(int32_t tile_m, int32_t tile_n) {
  if (!is_pow2(tile_m) || !is_pow2(tile_n) || tile_m < 16 || tile_n < 16 || tile_m > 1024 ||
      tile_n > 1024)
    return fail(HLA_ERR_UNSUPPORTED, "tiles %dx%d must be powers of two in [16, 1024]", tile_m, tile_n);
  return HLA_OK;
}

hla_status check_tensor_args(const void *a, const char *name) {
  if (!a) return fail(HLA_ERR_INVALID_ARG, "%s is NULL", name);
  if (!aligned(a, 16)) return fail(HLA_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return HLA_OK;
}

bool overlaps(const void *a, int64_t na, const void *b, int64_t nb) {
  const char *x = static_cast<const char *>(a), *y = static_cast<const char *>(b);
  return x < y + nb && y < x + na;
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float *g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on the current device, looked up once per
// device (with that device current) and kept. The stream, if given, must
// belong to the current device.
hla_status scratch_on_current_device(hipStream_t stream, float **ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(HLA_ERR_UNSUPPORTED, "device %d beyond the %d this library tracks", dev, kMaxDevices);
  if (stream) {
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return hip_status(e, "hipStreamGetDevice");
    if (sdev != dev)
      return fail(HLA_ERR_INVALID_ARG, "stream belongs to device %d, the current device is %d", (int)sdev, dev);
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(HLA_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = static_cast<float *>(p);
  }
  *ptr = g_scratch_ptr[dev];
  return HLA_OK;
}

}  // namespace

extern "C" {

const char *hla_last_error(void) { return g_last_error.c_str(); }

const char *hla_version(void) { return "libhla 0.1 (gfx950)"; }

static hla_status check_hilbert(int32_t H, int32_t W, const int32_t *order, const int32_t *rank) {
  if (H < 1 || W < 1) return fail(HLA_ERR_INVALID_ARG, "grid %dx%d must be positive", H, W);
  if (H > (1 << 15) || W > (1 << 15))
    return fail(HLA_ERR_UNSUPPORTED, "Hilbert order needs H, W <= 32768 (got %dx%d)", H, W);
  if (order && !aligned(order, 4)) return fail(HLA_ERR_INVALID_ARG, "order is not 4-byte aligned");
  if (rank && !aligned(rank, 4)) return fail(HLA_ERR_INVALID_ARG, "rank is not 4-byte aligned");
  if (order && rank && overlaps(order, (int64_t)H * W * 4, rank, (int64_t)H * W * 4))
    return fail(HLA_ERR_INVALID_ARG, "order and rank overlap");
  return HLA_OK;
}

hla_status hla_hilbert_perm(int32_t H, int32_t W, int32_t *order, int32_t *rank,
                            hla_stream_t stream) {
  hla_status st = check_hilbert(H, W, order, rank);
  if (st != HLA_OK) return st;
  if (!order && !rank) return HLA_OK;
  if (H == W && is_pow2(H))
    return hip_status(hla::launch_hilbert_perm(H, order, rank, (hipStream_t)stream), "hla_hilbert_perm");
  return hip_status(hla::launch_hilbert_grid(H, W, order, rank, (hipStream_t)stream), "hla_hilbert_perm");
}

static hla_status permute(const void *src, void *dst, const int32_t *order, int64_t B,
                          int64_t heads, int64_t N, int64_t d, hla_dtype dt,
                          hla_stream_t stream, bool scatter, const char *name) {
  hla_status st;
  if ((st = check_tensor_args(src, "src")) != HLA_OK) return st;
  if ((st = check_tensor_args(dst, "dst")) != HLA_OK) return st;
  if (!order) return fail(HLA_ERR_INVALID_ARG, "order is NULL");
  if (!aligned(order, 4)) return fail(HLA_ERR_INVALID_ARG, "order is not 4-byte aligned");
  if (B <= 0 || heads <= 0 || N <= 0 || d <= 0)
    return fail(HLA_ERR_INVALID_ARG, "sizes must be positive (B=%lld heads=%lld N=%lld d=%lld)",
                (long long)B, (long long)heads, (long long)N, (long long)d);
  const int64_t es = dtype_size(dt);
  if (!es) return fail(HLA_ERR_INVALID_ARG, "unknown dtype %d", (int)dt);
  const int64_t row = d * es;
  if (row % 4) return fail(HLA_ERR_UNSUPPORTED, "row of %lld bytes is not a multiple of 4", (long long)row);
  if (N > kMaxI32 || N * (row / 4) > kMaxI32 / 2)
    return fail(HLA_ERR_UNSUPPORTED, "N * row exceeds 2^30 words per (b, head) slice");
  if (B * heads > (1LL << 40)) return fail(HLA_ERR_UNSUPPORTED, "B * heads too large");
  const char *s = static_cast<const char *>(src);
  const char *e = s + B * heads * N * row;
  const char *o = static_cast<const char *>(dst);
  if (o < e && s < o + B * heads * N * row) return fail(HLA_ERR_INVALID_ARG, "src and dst overlap");
  return hip_status(hla::launch_permute(src, dst, order, B * heads, N, row, scatter, (hipStream_t)stream),
                    name);
}

hla_status hla_gather(const void *src, void *dst, const int32_t *order, int64_t B,
                      int64_t heads, int64_t N, int64_t d, hla_dtype dtype,
                      hla_stream_t stream) {
  return permute(src, dst, order, B, heads, N, d, dtype, stream, false, "hla_gather");
}

hla_status hla_scatter(const void *src, void *dst, const int32_t *order, int64_t B,
                       int64_t heads, int64_t N, int64_t d, hla_dtype dtype,
                       hla_stream_t stream) {
  return permute(src, dst, order, B, heads, N, d, dtype, stream, true, "hla_scatter");
}

hla_status hla_block_mask_dims(const hla_pattern_desc *pat, int32_t tile_m, int32_t tile_n,
                               int32_t *n_qtiles, int32_t *n_ktiles) {
  hla_status st;
  if ((st = check_pattern(pat)) != HLA_OK) return st;
  if ((st = check_tiles(tile_m, tile_n)) != HLA_OK) return st;
  const int64_t N = (int64_t)pat->H * pat->W;
  if (n_qtiles) *n_qtiles = (int32_t)((N + tile_m - 1) / tile_m);
  if (n_ktiles) *n_ktiles = (int32_t)((N + tile_n - 1) / tile_n);
  return HLA_OK;
}

// Validates a block mask for building and fills its host fields (N, n_qtiles,
// n_ktiles); *with_cols tells whether the transposed lists are asked for.
static hla_status check_block_mask(hla_block_mask *mask, bool *with_cols) {
  if (!mask) return fail(HLA_ERR_INVALID_ARG, "mask is NULL");
  int32_t nq = 0, nk = 0;
  hla_status st = hla_block_mask_dims(&mask->pat, mask->tile_m, mask->tile_n, &nq, &nk);
  if (st != HLA_OK) return st;
  if ((int64_t)nq * nk > kMaxI32) return fail(HLA_ERR_UNSUPPORTED, "tile grid %d x %d too large", nq, nk);
  int32_t *arrs[4] = {mask->n_full, mask->full_idx, mask->n_part, mask->part_idx};
  const char *names[4] = {"n_full", "full_idx", "n_part", "part_idx"};
  for (int i = 0; i < 4; ++i) {
    if (!arrs[i]) return fail(HLA_ERR_INVALID_ARG, "mask->%s is NULL", names[i]);
    if (!aligned(arrs[i], 4)) return fail(HLA_ERR_INVALID_ARG, "mask->%s is not 4-byte aligned", names[i]);
  }
  if (mask->totals && !aligned(mask->totals, 4))
    return fail(HLA_ERR_INVALID_ARG, "mask->totals is not 4-byte aligned");
  int32_t *cols[4] = {mask->n_full_t, mask->full_idx_t, mask->n_part_t, mask->part_idx_t};
  const char *cnames[4] = {"n_full_t", "full_idx_t", "n_part_t", "part_idx_t"};
  const int nset = (cols[0] != nullptr) + (cols[1] != nullptr) + (cols[2] != nullptr) +
                   (cols[3] != nullptr);
  if (nset != 0 && nset != 4)
    return fail(HLA_ERR_INVALID_ARG, "set all four transposed-list pointers or none");
  for (int i = 0; i < 4 && nset; ++i)
    if (!aligned(cols[i], 4)) return fail(HLA_ERR_INVALID_ARG, "mask->%s is not 4-byte aligned", cnames[i]);
  mask->N = mask->pat.H * mask->pat.W;
  mask->n_qtiles = nq;
  mask->n_ktiles = nk;
  *with_cols = nset == 4;
  return HLA_OK;
}

hla_status hla_build_block_mask(hla_block_mask *mask, hla_stream_t stream) {
  bool with_cols = false;
  hla_status st = check_block_mask(mask, &with_cols);
  if (st != HLA_OK) return st;
  const hla::PatternArgs pa = hla::make_pattern_args(mask->pat);
  const hla::BlockLists rows = {mask->n_full, mask->full_idx, mask->n_part, mask->part_idx};
  const hla::BlockLists tcols = {mask->n_full_t, mask->full_idx_t, mask->n_part_t, mask->part_idx_t};
  return hip_status(hla::launch_block_mask(pa, mask->tile_m, mask->tile_n, mask->n_qtiles,
                                           mask->n_ktiles, rows, with_cols ? &tcols : nullptr,
                                           mask->totals, (hipStream_t)stream),
                    "hla_build_block_mask");
}

hla_status hla_build_path_and_mask(int32_t H, int32_t W, int32_t *order, int32_t *rank,
                                   hla_block_mask *mask, hla_stream_t stream) {
  hla_status st = check_hilbert(H, W, order, rank);
  if (st != HLA_OK) return st;
  bool with_cols = false;
  if ((st = check_block_mask(mask, &with_cols)) != HLA_OK) return st;
  if (mask->pat.H != H || mask->pat.W != W)
    return fail(HLA_ERR_INVALID_ARG, "the mask's pattern is on a %dx%d grid, the path on %dx%d",
                mask->pat.H, mask->pat.W, H, W);
  const int64_t nb = (int64_t)H * W * 4;
  int32_t *outs[2] = {order, rank};
  const char *onames[2] = {"order", "rank"};
  int32_t *arrs[8] = {mask->n_full, mask->full_idx, mask->n_part, mask->part_idx,
                      mask->n_full_t, mask->full_idx_t, mask->n_part_t, mask->part_idx_t};
  const int64_t alen[8] = {(int64_t)mask->n_qtiles * 4, (int64_t)mask->n_qtiles * mask->n_ktiles * 4,
                           (int64_t)mask->n_qtiles * 4, (int64_t)mask->n_qtiles * mask->n_ktiles * 4,
                           (int64_t)mask->n_ktiles * 4, (int64_t)mask->n_qtiles * mask->n_ktiles * 4,
                           (int64_t)mask->n_ktiles * 4, (int64_t)mask->n_qtiles * mask->n_ktiles * 4};
  for (int o = 0; o < 2; ++o) {
    if (!outs[o]) continue;
    for (int i = 0; i < 8; ++i)
      if (arrs[i] && overlaps(outs[o], nb, arrs[i], alen[i]))
        return fail(HLA_ERR_INVALID_ARG, "%s overlaps the mask's arrays", onames[o]);
    if (mask->totals && overlaps(outs[o], nb, mask->totals, 8))
      return fail(HLA_ERR_INVALID_ARG, "%s overlaps mask->totals", onames[o]);
  }
  const hla::PatternArgs pa = hla::make_pattern_args(mask->pat);
  const hla::BlockLists rows = {mask->n_full, mask->full_idx, mask->n_part, mask->part_idx};
  const hla::BlockLists tcols = {mask->n_full_t, mask->full_idx_t, mask->n_part_t, mask->part_idx_t};
  const hipStream_t s = (hipStream_t)stream;
  if (H == W && is_pow2(H) && H >= 4 && (order || rank))
    return hip_status(hla::launch_path_and_mask(H, order, rank, pa, mask->tile_m, mask->tile_n,
                                                mask->n_qtiles, mask->n_ktiles, rows,
                                                with_cols ? &tcols : nullptr, mask->totals, s),
                      "hla_build_path_and_mask");
  if (order || rank) {
    const hipError_t e = H == W && is_pow2(H) ? hla::launch_hilbert_perm(H, order, rank, s)
                                              : hla::launch_hilbert_grid(H, W, order, rank, s);
    if (e != hipSuccess) return hip_status(e, "hla_build_path_and_mask");
  }
  return hip_status(hla::launch_block_mask(pa, mask->tile_m, mask->tile_n, mask->n_qtiles,
                                           mask->n_ktiles, rows, with_cols ? &tcols : nullptr,
                                           mask->totals, s),
                    "hla_build_path_and_mask");
}

}  // extern "C"

namespace {

// Checks shared by the attention passes: the mask, sizes, dtype, scale and the
// supported shapes. Pointers are checked by the callers.
// (need_lists = false: the kernel classifies its own tiles, so the mask's arrays
// are not read.)
hla_status check_attn(const hla_block_mask *mask, int64_t B, int64_t heads, int64_t N,
                      int64_t d, hla_dtype dtype, float scale, bool need_lists = true) {
  hla_status st;
  if (!mask) return fail(HLA_ERR_INVALID_ARG, "mask is NULL");
  if (need_lists && (!mask->n_full || !mask->full_idx || !mask->n_part || !mask->part_idx))
    return fail(HLA_ERR_INVALID_ARG, "mask arrays are NULL (build the mask first)");
  if (B <= 0 || heads <= 0 || N <= 0 || d <= 0)
    return fail(HLA_ERR_INVALID_ARG, "sizes must be positive");
  if (!(scale > 0.f) || scale > 1e30f) return fail(HLA_ERR_INVALID_ARG, "scale must be positive and finite");
  if ((st = check_pattern(&mask->pat)) != HLA_OK) return st;
  if ((st = check_tiles(mask->tile_m, mask->tile_n)) != HLA_OK) return st;
  const int64_t mN = (int64_t)mask->pat.H * mask->pat.W;
  if (mask->N != mN || N != mN || mask->n_qtiles != (mN + mask->tile_m - 1) / mask->tile_m ||
      mask->n_ktiles != (mN + mask->tile_n - 1) / mask->tile_n)
    return fail(HLA_ERR_INVALID_ARG, "mask was built for N = %d, attention has N = %lld",
                mask->N, (long long)N);
  if (dtype != HLA_F32 && dtype != HLA_BF16) return fail(HLA_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
  if (d != 32 && d != 64) return fail(HLA_ERR_UNSUPPORTED, "head_dim %lld (supported: 32, 64)", (long long)d);
  if (mask->tile_n != 64 || (mask->tile_m != 64 && mask->tile_m != 128))
    return fail(HLA_ERR_UNSUPPORTED, "tile %dx%d (supported: 64x64, 128x64)", mask->tile_m, mask->tile_n);
  if (N * d > (1LL << 30)) return fail(HLA_ERR_UNSUPPORTED, "N * d exceeds 2^30 per (b, head)");
  const int64_t BH = B * heads;
  if (BH * mask->n_qtiles > kMaxI32 || BH * mask->n_ktiles > kMaxI32 || BH * N > kMaxI32)
    return fail(HLA_ERR_UNSUPPORTED, "grid too large");
  return HLA_OK;
}

}  // namespace

extern "C" {

static hla_status attn_fwd(const void *q, const void *k, const void *v, const int32_t *order,
                           const float *rpb, int mode, const hla_block_mask *mask, void *out,
                           float *lse, int64_t B, int64_t heads, int64_t N, int64_t d,
                           hla_dtype dtype, float scale, hla_stream_t stream, const char *name) {
  hla_status st;
  if ((st = check_tensor_args(q, "q")) != HLA_OK) return st;
  if ((st = check_tensor_args(k, "k")) != HLA_OK) return st;
  if ((st = check_tensor_args(v, "v")) != HLA_OK) return st;
  if ((st = check_tensor_args(out, "out")) != HLA_OK) return st;
  if (lse && !aligned(lse, 4)) return fail(HLA_ERR_INVALID_ARG, "lse is not 4-byte aligned");
  if ((st = check_attn(mask, B, heads, N, d, dtype, scale, mode != hla::ATTN_HILBERT)) != HLA_OK)
    return st;
  const int64_t BH = B * heads;
  const int64_t bytes = BH * N * d * dtype_size(dtype);
  for (const void *in : {q, k, v})
    if (overlaps(out, bytes, in, bytes)) return fail(HLA_ERR_INVALID_ARG, "out overlaps an input");
  if (lse && overlaps(lse, BH * N * 4, out, bytes))
    return fail(HLA_ERR_INVALID_ARG, "lse overlaps out");
  hla::AttnArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.lse = lse;
  a.order = order;
  a.rpb = rpb;
  a.mode = mode;
  a.n_full = mask->n_full;
  a.full_idx = mask->full_idx;
  a.n_part = mask->n_part;
  a.part_idx = mask->part_idx;
  a.BH = (int32_t)BH;
  a.heads = (int32_t)heads;
  a.N = (int32_t)N;
  a.n_qtiles = mask->n_qtiles;
  a.n_ktiles = mask->n_ktiles;
  a.scale = scale;
  a.scale_log2 = (float)((double)scale * 1.4426950408889634074);
  a.pat = hla::make_pattern_args(mask->pat);
  a.lg = 0;
  a.hgroups = (int32_t)BH;
  while ((1 << a.lg) < mask->pat.W) ++a.lg;
  hipError_t e = dtype == HLA_BF16
                     ? hla::launch_attn_bf16(a, (int)d, mask->tile_m, mask->tile_n, (hipStream_t)stream)
                     : hla::launch_attn_f32(a, (int)d, mask->tile_m, mask->tile_n, (hipStream_t)stream);
  return hip_status(e, name);
}

hla_status hla_attn_fwd(const void *q, const void *k, const void *v, const hla_block_mask *mask,
                        void *out, float *lse, int64_t B, int64_t heads, int64_t N, int64_t d,
                        hla_dtype dtype, float scale, hla_stream_t stream) {
  return attn_fwd(q, k, v, nullptr, nullptr, hla::ATTN_PLAIN, mask, out, lse, B, heads, N, d,
                  dtype, scale, stream, "hla_attn_fwd");
}

hla_status hla_attn_fwd_perm(const void *q, const void *k, const void *v, const int32_t *order,
                             const hla_block_mask *mask, void *out, float *lse, int64_t B,
                             int64_t heads, int64_t N, int64_t d, hla_dtype dtype, float scale,
                             hla_stream_t stream) {
  if (!order) return fail(HLA_ERR_INVALID_ARG, "order is NULL");
  if (!aligned(order, 16)) return fail(HLA_ERR_INVALID_ARG, "order is not 16-byte aligned");
  for (const void *t : {q, k, v, (const void *)out})
    if (t && overlaps(order, N * 4, t, B * heads * N * d * dtype_size(dtype)))
      return fail(HLA_ERR_INVALID_ARG, "order overlaps a tensor");
  return attn_fwd(q, k, v, order, nullptr, hla::ATTN_GATHER, mask, out, lse, B, heads, N, d,
                  dtype, scale, stream, "hla_attn_fwd_perm");
}

hla_status hla_attn_fwd_hilbert(const void *q, const void *k, const void *v,
                                const hla_pattern_desc *pat, int32_t tile_m, int32_t tile_n,
                                void *out, float *lse, int64_t B, int64_t heads, int64_t N,
                                int64_t d, hla_dtype dtype, float scale, hla_stream_t stream) {
  hla_status st;
  if (!pat) return fail(HLA_ERR_INVALID_ARG, "pat is NULL");
  if ((st = check_pattern(pat)) != HLA_OK) return st;
  if (pat->pattern != HLA_HILBERT_WINDOW && pat->pattern != HLA_HILBERT_SLIDE &&
      pat->pattern != HLA_HILBERT_NEIGHBORHOOD && pat->pattern != HLA_HILBERT_SHIFTED_WINDOW)
    return fail(HLA_ERR_UNSUPPORTED, "hla_attn_fwd_hilbert takes the Hilbert patterns (got %d)",
                (int)pat->pattern);
  if (pat->H != pat->W || pat->W < 8 || (pat->W & (pat->W - 1)) != 0)
    return fail(HLA_ERR_UNSUPPORTED, "hla_attn_fwd_hilbert needs a 2^k x 2^k grid with side >= 8 "
                "(got %d x %d)", pat->H, pat->W);
  if (dtype != HLA_BF16) return fail(HLA_ERR_UNSUPPORTED, "hla_attn_fwd_hilbert takes bf16 only");
  if ((st = check_tiles(tile_m, tile_n)) != HLA_OK) return st;
  hla_block_mask m;
  std::memset(&m, 0, sizeof(m));
  m.N = pat->H * pat->W;
  m.tile_m = tile_m;
  m.tile_n = tile_n;
  m.n_qtiles = (m.N + tile_m - 1) / tile_m;
  m.n_ktiles = (m.N + tile_n - 1) / tile_n;
  m.pat = *pat;
  return attn_fwd(q, k, v, nullptr, nullptr, hla::ATTN_HILBERT, &m, out, lse, B, heads, N, d,
                  dtype, scale, stream, "hla_attn_fwd_hilbert");
}

hla_status hla_attn_fwd_rpb(const void *q, const void *k, const void *v, const int32_t *order,
                            const float *rpb, const hla_block_mask *mask, void *out, float *lse,
                            int64_t B, int64_t heads, int64_t N, int64_t d, hla_dtype dtype,
                            float scale, hla_stream_t stream) {
  if (!order) return fail(HLA_ERR_INVALID_ARG, "order is NULL");
  if (!aligned(order, 16)) return fail(HLA_ERR_INVALID_ARG, "order is not 16-byte aligned");
  if (!rpb) return fail(HLA_ERR_INVALID_ARG, "rpb is NULL");
  if (!aligned(rpb, 4)) return fail(HLA_ERR_INVALID_ARG, "rpb is not 4-byte aligned");
  if (!mask) return fail(HLA_ERR_INVALID_ARG, "mask is NULL");
  if (heads <= 0 || heads > (1 << 20)) return fail(HLA_ERR_INVALID_ARG, "heads must be in [1, 2^20]");
  const int64_t tab = (2LL * mask->pat.H - 1) * (2LL * mask->pat.W - 1);
  if (mask->pat.H <= 0 || mask->pat.W <= 0 || tab * heads > kMaxI32)
    return fail(HLA_ERR_UNSUPPORTED, "bias table of %lld entries per head is too large", (long long)tab);
  const int64_t tbytes = B * heads * N * d * dtype_size(dtype);
  for (const void *t : {q, k, v, (const void *)out}) {
    if (t && overlaps(order, N * 4, t, tbytes)) return fail(HLA_ERR_INVALID_ARG, "order overlaps a tensor");
    if (t && overlaps(rpb, tab * heads * 4, t, tbytes)) return fail(HLA_ERR_INVALID_ARG, "rpb overlaps a tensor");
  }
  if (lse && overlaps(rpb, tab * heads * 4, lse, B * heads * N * 4))
    return fail(HLA_ERR_INVALID_ARG, "rpb overlaps lse");
  return attn_fwd(q, k, v, order, rpb, hla::ATTN_RPB, mask, out, lse, B, heads, N, d, dtype, scale,
                  stream, "hla_attn_fwd_rpb");
}

// stats == nullptr: the row statistics go to the library's own `scratch` array
// (hla_attn_bwd_noalloc); the public entry points with a stats argument reject
// a null one before calling this.
static hla_status attn_bwd(const void *q, const void *k, const void *v, const void *out,
                           const void *dout, const float *lse, const int32_t *order,
                           const hla_block_mask *mask, void *dq, void *dk, void *dv, float *stats,
                           int64_t B, int64_t heads, int64_t N, int64_t d, hla_dtype dtype,
                           float scale, hla_stream_t stream, const char *name) {
  hla_status st;
  const bool own_stats = stats == nullptr;
  const void *ins[5] = {q, k, v, out, dout};
  const char *in_names[5] = {"q", "k", "v", "out", "dout"};
  for (int i = 0; i < 5; ++i)
    if ((st = check_tensor_args(ins[i], in_names[i])) != HLA_OK) return st;
  void *outs[3] = {dq, dk, dv};
  const char *out_names[3] = {"dq", "dk", "dv"};
  for (int i = 0; i < 3; ++i)
    if ((st = check_tensor_args(outs[i], out_names[i])) != HLA_OK) return st;
  if ((st = check_tensor_args(lse, "lse")) != HLA_OK) return st;
  if (!own_stats && (st = check_tensor_args(stats, "stats")) != HLA_OK) return st;
  if ((st = check_attn(mask, B, heads, N, d, dtype, scale)) != HLA_OK) return st;
  if (!mask->n_full_t || !mask->full_idx_t || !mask->n_part_t || !mask->part_idx_t)
    return fail(HLA_ERR_INVALID_ARG, "the mask has no transposed lists (set them before building it)");
  const int64_t BH = B * heads;
  const int64_t bytes = BH * N * d * dtype_size(dtype);
  if (own_stats && BH * N > kScratchRows)
    return fail(HLA_ERR_UNSUPPORTED, "B * heads * N = %lld rows exceeds the %lld the library's "
                "row-statistics array holds (use hla_attn_bwd with a stats workspace)",
                (long long)(BH * N), (long long)kScratchRows);
  for (int i = 0; i < 3; ++i) {
    for (int j = 0; j < 5; ++j)
      if (overlaps(outs[i], bytes, ins[j], bytes))
        return fail(HLA_ERR_INVALID_ARG, "%s overlaps %s", out_names[i], in_names[j]);
    for (int j = i + 1; j < 3; ++j)
      if (overlaps(outs[i], bytes, outs[j], bytes))
        return fail(HLA_ERR_INVALID_ARG, "%s overlaps %s", out_names[i], out_names[j]);
    if (!own_stats && overlaps(outs[i], bytes, stats, BH * N * 8))
      return fail(HLA_ERR_INVALID_ARG, "%s overlaps stats", out_names[i]);
  }
  if (!own_stats) {
    for (int j = 0; j < 5; ++j)
      if (overlaps(stats, BH * N * 8, ins[j], bytes))
        return fail(HLA_ERR_INVALID_ARG, "stats overlaps %s", in_names[j]);
    if (overlaps(stats, BH * N * 8, lse, BH * N * 4))
      return fail(HLA_ERR_INVALID_ARG, "stats overlaps lse");
  }
  if (order) {
    for (int i = 0; i < 3; ++i)
      if (overlaps(order, N * 4, outs[i], bytes)) return fail(HLA_ERR_INVALID_ARG, "order overlaps %s", out_names[i]);
    if (!own_stats && overlaps(order, N * 4, stats, BH * N * 8))
      return fail(HLA_ERR_INVALID_ARG, "order overlaps stats");
  }
  // every argument is valid: only now look up the library's array (a HIP call)
  if (own_stats && (st = scratch_on_current_device((hipStream_t)stream, &stats)) != HLA_OK) return st;
  hla::AttnBwdArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.out = out;
  a.dout = dout;
  a.lse = lse;
  a.stats = stats;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.order = order;
  a.n_full = mask->n_full;
  a.full_idx = mask->full_idx;
  a.n_part = mask->n_part;
  a.part_idx = mask->part_idx;
  a.n_full_t = mask->n_full_t;
  a.full_idx_t = mask->full_idx_t;
  a.n_part_t = mask->n_part_t;
  a.part_idx_t = mask->part_idx_t;
  a.BH = (int32_t)BH;
  a.N = (int32_t)N;
  a.n_qtiles = mask->n_qtiles;
  a.n_ktiles = mask->n_ktiles;
  a.scale = scale;
  a.scale_log2 = (float)((double)scale * 1.4426950408889634074);
  a.pat = hla::make_pattern_args(mask->pat);
  a.hgroups = (int32_t)BH;
  hipError_t e =
      dtype == HLA_BF16
          ? hla::launch_attn_bwd_bf16(a, (int)d, mask->tile_m, mask->tile_n, (hipStream_t)stream)
          : hla::launch_attn_bwd_f32(a, (int)d, mask->tile_m, mask->tile_n, (hipStream_t)stream);
  return hip_status(e, name);
}

hla_status hla_attn_bwd(const void *q, const void *k, const void *v, const void *out,
                        const void *dout, const float *lse, const hla_block_mask *mask, void *dq,
                        void *dk, void *dv, float *stats, int64_t B, int64_t heads, int64_t N,
                        int64_t d, hla_dtype dtype, float scale, hla_stream_t stream) {
  if (!stats) return fail(HLA_ERR_INVALID_ARG, "stats is NULL");
  return attn_bwd(q, k, v, out, dout, lse, nullptr, mask, dq, dk, dv, stats, B, heads, N, d, dtype,
                  scale, stream, "hla_attn_bwd");
}

hla_status hla_attn_bwd_perm(const void *q, const void *k, const void *v, const void *out,
                             const void *dout, const float *lse, const int32_t *order,
                             const hla_block_mask *mask, void *dq, void *dk, void *dv,
                             float *stats, int64_t B, int64_t heads, int64_t N, int64_t d,
                             hla_dtype dtype, float scale, hla_stream_t stream) {
  if (!order) return fail(HLA_ERR_INVALID_ARG, "order is NULL");
  if (!aligned(order, 16)) return fail(HLA_ERR_INVALID_ARG, "order is not 16-byte aligned");
  if (!stats) return fail(HLA_ERR_INVALID_ARG, "stats is NULL");
  return attn_bwd(q, k, v, out, dout, lse, order, mask, dq, dk, dv, stats, B, heads, N, d, dtype,
                  scale, stream, "hla_attn_bwd_perm");
}

hla_status hla_attn_bwd_noalloc(const void *q, const void *k, const void *v, const void *out,
                                const void *dout, const float *lse, const hla_block_mask *mask,
                                void *dq, void *dk, void *dv, int64_t B, int64_t heads, int64_t N,
                                int64_t d, hla_dtype dtype, float scale, hla_stream_t stream) {
  return attn_bwd(q, k, v, out, dout, lse, nullptr, mask, dq, dk, dv, nullptr, B, heads, N, d,
                  dtype, scale, stream, "hla_attn_bwd_noalloc");
}

static hla_status qkv_proj(const void *x, const void *w_qkv, const int32_t *order, void *q,
                           void *k, void *v, int64_t B, int64_t N, int64_t heads, int64_t d,
                           hla_stream_t stream, const char *name) {
  hla_status st;
  if ((st = check_tensor_args(x, "x")) != HLA_OK) return st;
  if ((st = check_tensor_args(w_qkv, "w_qkv")) != HLA_OK) return st;
  if ((st = check_tensor_args(q, "q")) != HLA_OK) return st;
  if ((st = check_tensor_args(k, "k")) != HLA_OK) return st;
  if ((st = check_tensor_args(v, "v")) != HLA_OK) return st;
  if (B <= 0 || N <= 0 || heads <= 0 || d <= 0) return fail(HLA_ERR_INVALID_ARG, "sizes must be positive");
  if (d != 32 && d != 64) return fail(HLA_ERR_UNSUPPORTED, "head_dim %lld (supported: 32, 64)", (long long)d);
  const int64_t C = heads * d;
  if (C % 64 || C > 512) return fail(HLA_ERR_UNSUPPORTED, "C = heads*d = %lld must be a multiple of 64, <= 512", (long long)C);
  if (B * N * C > (1LL << 31) - 1 || B * N > (1LL << 31) - 256)
    return fail(HLA_ERR_UNSUPPORTED, "B * N * C exceeds 2^31");
  return hip_status(hla::launch_qkv_proj(x, w_qkv, order, q, k, v, B, N, heads, d, (hipStream_t)stream),
                    name);
}

static hla_status out_proj(const void *o, const void *w_proj, const int32_t *order, void *y,
                           int64_t B, int64_t N, int64_t heads, int64_t d, int64_t c_out,
                           hla_stream_t stream, const char *name) {
  hla_status st;
  if ((st = check_tensor_args(o, "o")) != HLA_OK) return st;
  if ((st = check_tensor_args(w_proj, "w_proj")) != HLA_OK) return st;
  if ((st = check_tensor_args(y, "y")) != HLA_OK) return st;
  if (B <= 0 || N <= 0 || heads <= 0 || d <= 0 || c_out <= 0)
    return fail(HLA_ERR_INVALID_ARG, "sizes must be positive");
  if (d != 32 && d != 64) return fail(HLA_ERR_UNSUPPORTED, "head_dim %lld (supported: 32, 64)", (long long)d);
  const int64_t C = heads * d;
  if (C % 64 || C > 512) return fail(HLA_ERR_UNSUPPORTED, "C = heads*d = %lld must be a multiple of 64, <= 512", (long long)C);
  if (c_out % 64) return fail(HLA_ERR_UNSUPPORTED, "c_out = %lld must be a multiple of 64", (long long)c_out);
  if (B * N * (C > c_out ? C : c_out) > (1LL << 31) - 1 || B * N > (1LL << 31) - 256)
    return fail(HLA_ERR_UNSUPPORTED, "B * N * C exceeds 2^31");
  return hip_status(hla::launch_out_proj(o, w_proj, order, y, B, N, heads, d, c_out, (hipStream_t)stream),
                    name);
}

hla_status hla_qkv_proj(const void *x, const void *w_qkv, void *q, void *k, void *v, int64_t B,
                        int64_t N, int64_t heads, int64_t d, hla_stream_t stream) {
  return qkv_proj(x, w_qkv, nullptr, q, k, v, B, N, heads, d, stream, "hla_qkv_proj");
}

hla_status hla_qkv_proj_perm(const void *x, const void *w_qkv, const int32_t *order, void *q,
                             void *k, void *v, int64_t B, int64_t N, int64_t heads, int64_t d,
                             hla_stream_t stream) {
  if (!order) return fail(HLA_ERR_INVALID_ARG, "order is null");
  if (!aligned(order, 16)) return fail(HLA_ERR_INVALID_ARG, "order is not 16-byte aligned");
  return qkv_proj(x, w_qkv, order, q, k, v, B, N, heads, d, stream, "hla_qkv_proj_perm");
}

hla_status hla_out_proj(const void *o, const void *w_proj, void *y, int64_t B, int64_t N,
                        int64_t heads, int64_t d, int64_t c_out, hla_stream_t stream) {
  return out_proj(o, w_proj, nullptr, y, B, N, heads, d, c_out, stream, "hla_out_proj");
}

hla_status hla_out_proj_perm(const void *o, const void *w_proj, const int32_t *order, void *y,
                             int64_t B, int64_t N, int64_t heads, int64_t d, int64_t c_out,
                             hla_stream_t stream) {
  if (!order) return fail(HLA_ERR_INVALID_ARG, "order is null");
  if (!aligned(order, 16)) return fail(HLA_ERR_INVALID_ARG, "order is not 16-byte aligned");
  return out_proj(o, w_proj, order, y, B, N, heads, d, c_out, stream, "hla_out_proj_perm");
}

}  // extern "C"
