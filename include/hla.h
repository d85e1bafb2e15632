/*
 * hla.h - C ABI of libhla: Hilbert-guided block-sparse local attention on
 * AMD Instinct MI355X (gfx950).
 *
 * Method: Li & Xu, "Hilbert-Guided Sparse Local Attention" (arXiv 2511.05832).
 * Image tokens are reordered along a Hilbert curve, windows or slide bands are
 * formed on the reordered 1-D sequence (Sec. 3.1), and a block-sparse attention
 * forward pass skips empty tiles, runs full tiles unmasked and masks only
 * partial tiles (Sec. 3.1, block types; Eq. 1).
 *
 * Conventions shared by every entry point
 *  - Every call returns hla_status; HLA_OK is 0. No call throws or aborts.
 *  - Arguments are validated on the host before any HIP call. On a status other
 *    than HLA_OK nothing has been enqueued and no output has been written; the
 *    text of the error is available from hla_last_error() on the same thread.
 *  - Device pointers are plain device addresses owned by the caller. The library
 *    allocates and frees no device memory; its only device memory of its own is
 *    the array of hla_attn_bwd_noalloc, part of its code object.
 *  - Work is enqueued on the caller's stream (NULL = the default stream) and the
 *    calls never synchronise, so they may be captured into a HIP graph.
 *  - Tensors are dense and contiguous, innermost dimension last:
 *      attention tensors  [B, heads, N, d]
 *      layer activations  [B, N, C]
 *  - Base addresses of tensors must be 16-byte aligned; index arrays 4-byte.
 *  - Element types: HLA_F32 (IEEE binary32) and HLA_BF16 (bfloat16 stored as
 *    uint16). Conversions to bf16 round to nearest even.
 *  - Status HLA_ERR_INVALID_ARG: a null or misaligned pointer, a non-positive
 *    or inconsistent size. HLA_ERR_UNSUPPORTED: valid but outside what this
 *    build implements (listed per call). HLA_ERR_HIP: a HIP launch failed; the
 *    HIP error text is in hla_last_error().
 *  - Thread safety: re-entrant. The global state is the per-thread error text
 *    and hla_attn_bwd_noalloc's per-device array. Calls that write the same
 *    buffers on different streams race.
 */
#ifndef HLA_H
#define HLA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t *hla_stream_t; /* a hipStream_t */

typedef enum {
  HLA_OK = 0,
  HLA_ERR_INVALID_ARG = 1,
  HLA_ERR_UNSUPPORTED = 2,
  HLA_ERR_HIP = 3
} hla_status;

typedef enum { HLA_F32 = 0, HLA_BF16 = 1 } hla_dtype;

/*
 * Attention patterns (Sec. 3.1-3.3). i, j are positions of a query and a key in
 * the sequence as stored. For the Hilbert patterns the sequence is in Hilbert
 * order (gathered with hla_gather); for the row-major patterns it is in
 * row-major order and a position t is the grid cell (r, c) = (t / W, t % W).
 *
 *  HLA_HILBERT_WINDOW      p0 = w:      floor(i/w) == floor(j/w)
 *                          (contiguous windows on the Hilbert sequence, HWA)
 *  HLA_HILBERT_SLIDE       p0 = h:      |i - j| <= h      (band, HSA)
 *  HLA_ROWMAJOR_WINDOW     p0, p1 = window rows, cols: same (r/p0, c/p1) cell (WSA)
 *  HLA_ROWMAJOR_SLIDE      p0, p1 = radius rows, cols: |r-r'| <= p0 && |c-c'| <= p1 (SA)
 *  HLA_HILBERT_NEIGHBORHOOD p0 = k: j in [s, s+k), s = clamp(i - k/2, 0, N-k) (HNA)
 *  HLA_ROWMAJOR_NEIGHBORHOOD p0, p1 = kernel rows, cols: the same clamp per axis (NA2D)
 *  HLA_HILBERT_SHIFTED_WINDOW p0 = w, p1 = s: floor((i+w-s)/w) == floor((j+w-s)/w)
 *                          (windows moved by s along the sequence; the pairs a
 *                          cyclic shift would join across the ends are masked, HSWA)
 */
typedef enum {
  HLA_HILBERT_WINDOW = 0,
  HLA_HILBERT_SLIDE = 1,
  HLA_ROWMAJOR_WINDOW = 2,
  HLA_ROWMAJOR_SLIDE = 3,
  HLA_HILBERT_NEIGHBORHOOD = 4,
  HLA_ROWMAJOR_NEIGHBORHOOD = 5,
  HLA_HILBERT_SHIFTED_WINDOW = 6
} hla_pattern;

typedef struct {
  int32_t pattern; /* hla_pattern */
  int32_t H, W;    /* token grid; N = H * W */
  int32_t p0, p1;  /* pattern parameters, see hla_pattern */
} hla_pattern_desc;

/*
 * Block-sparse metadata (Sec. 3.1: full / partial / empty blocks; the paper's
 * engine keeps only this lightweight block metadata, Sec. 4.2).
 * The N x N score matrix is cut into tiles of tile_m query rows by tile_n key
 * columns: n_qtiles = ceil(N / tile_m), n_ktiles = ceil(N / tile_n). When a tile
 * size does not divide N (the paper's 56x56 grid at block 128, Tables 3 and 6)
 * the last tiles reach past N; their padded slots are never allowed, so such a
 * tile is partial or empty, never full. For query-tile row q:
 *   n_full[q]            number of full tiles
 *   full_idx[q*n_ktiles + t], t < n_full[q]: key-tile indices, ascending
 *   n_part[q], part_idx  the same for partial tiles
 * Unused list entries are -1. All four arrays are caller-owned device memory:
 * n_full, n_part hold n_qtiles int32; full_idx, part_idx hold
 * n_qtiles * n_ktiles int32 (hla_block_mask_dims gives the counts).
 * totals, if not NULL, is a device int32[2] that receives
 * {total full tiles, total partial tiles}.
 *
 * Optional transposed lists, read by the backward pass (hla_attn_bwd) to
 * accumulate key and value gradients per key tile. For key-tile column k:
 *   n_full_t[k]            number of full tiles in the column
 *   full_idx_t[k*n_qtiles + t], t < n_full_t[k]: query-tile indices, ascending
 *   n_part_t[k], part_idx_t  the same for partial tiles
 * n_full_t, n_part_t hold n_ktiles int32; full_idx_t, part_idx_t hold
 * n_ktiles * n_qtiles int32; unused entries are -1. Set all four or none
 * (NULL: not built).
 */
typedef struct {
  int32_t N, tile_m, tile_n, n_qtiles, n_ktiles;
  hla_pattern_desc pat;
  int32_t *n_full, *full_idx, *n_part, *part_idx;
  int32_t *totals;
  int32_t *n_full_t, *full_idx_t, *n_part_t, *part_idx_t;
} hla_block_mask;

/*
 * Hilbert index and its inverse (Sec. 3.1-3.2: the path P_(H,W) is computed
 * once per feature-map size and cached by the caller).
 * order[d] = row-major id (y*W + x) of the d-th cell on the curve;
 * rank[t]  = position of row-major token t on the curve (rank[order[d]] = d).
 * Curve: starts at cell (x,y) = (0,0), first step to (0,1), ends at (W-1,0).
 * Any other grid (the paper also uses 56x56, 96x96, 160x160 and 128x256
 * feature maps and does not say how its curve covers them): the curve on the
 * smallest 2^k x 2^k square holding the grid (grid at its (0,0) corner), with
 * the cells outside the grid left out, in the curve's order.
 * order, rank: device int32[H*W]; either may be NULL to skip it; they may not
 * overlap. INVALID_ARG unless H, W >= 1; UNSUPPORTED if H or W > 32768.
 */
hla_status hla_hilbert_perm(int32_t H, int32_t W, int32_t *order, int32_t *rank,
                            hla_stream_t stream);

/*
 * Gather into Hilbert order (the paper's "reshape" step, Sec. 4.2):
 *   dst[b,h,i,:] = src[b,h,order[i],:]  for i < N.
 * src, dst: [B, heads, N, d] of dtype, must not overlap. order: device int32[N],
 * a permutation of [0, N) (not checked; an out-of-range entry is undefined
 * behaviour). Any d >= 1 with d * sizeof(dtype) a multiple of 4.
 */
hla_status hla_gather(const void *src, void *dst, const int32_t *order,
                      int64_t B, int64_t heads, int64_t N, int64_t d,
                      hla_dtype dtype, hla_stream_t stream);

/*
 * Scatter back to row-major order (the inverse of hla_gather):
 *   dst[b,h,order[i],:] = src[b,h,i,:].
 * Same arguments and constraints as hla_gather.
 */
hla_status hla_scatter(const void *src, void *dst, const int32_t *order,
                       int64_t B, int64_t heads, int64_t N, int64_t d,
                       hla_dtype dtype, hla_stream_t stream);

/*
 * Host-only: tile-grid sizes of the block-sparse metadata (Sec. 3.1: the score
 * matrix cut into b_q x b_k blocks, each full, partial or empty), so the caller
 * can size the block-mask arrays: n_qtiles = ceil(N / tile_m), n_ktiles = ceil(N / tile_n),
 * N = H*W (any N; tiles may be ragged). Tile sizes are powers of two in
 * [16, 1024]. Pattern parameters must be >= 1
 * (slide radii and half-widths >= 0; neighbourhood kernels <= the grid extent).
 */
hla_status hla_block_mask_dims(const hla_pattern_desc *pat, int32_t tile_m,
                               int32_t tile_n, int32_t *n_qtiles,
                               int32_t *n_ktiles);

/*
 * Classify every (query tile, key tile) pair as full, partial or empty and write
 * the per-row ascending lists (Sec. 3.1). mask->pat, tile_m, tile_n select the
 * pattern and tiling; the call fills mask->N, n_qtiles, n_ktiles on the host
 * and the four device arrays (and totals) on the stream, plus the transposed
 * lists when their four pointers are set. It does not synchronise. The
 * classification is exact: for every pattern the class of a tile equals the
 * one obtained by counting its allowed elements.
 */
hla_status hla_build_block_mask(hla_block_mask *mask, hla_stream_t stream);

/*
 * hla_hilbert_perm and hla_build_block_mask in one call, for a step that builds
 * both: the path P_(H,W) (Sec. 3.2) and the block metadata of a pattern on the
 * same H x W grid (Sec. 3.1). On a 2^k x 2^k grid with k >= 2 the index and the
 * row lists come from a single launch (one graph node instead of two; the
 * transposed lists and the totals, if asked for, take their usual launches
 * after it); on any other grid the two calls' launches run in sequence. The
 * results equal hla_hilbert_perm followed by hla_build_block_mask bit for bit.
 * order, rank: as for hla_hilbert_perm (either or both may be NULL), not
 * overlapping any of the mask's arrays. mask: as for hla_build_block_mask, with
 * mask->pat on the same grid (pat.H == H, pat.W == W; else INVALID_ARG). Both are
 * validated before anything is enqueued; errors as the two calls'.
 */
hla_status hla_build_path_and_mask(int32_t H, int32_t W, int32_t *order, int32_t *rank,
                                   hla_block_mask *mask, hla_stream_t stream);

/*
 * Block-sparse attention forward (Sec. 3.1; Eq. 1's per-tile work). For every
 * (b, h) and query-tile row, walks only the listed key tiles: full tiles
 * without a mask, partial tiles with the element mask of mask->pat. Computes
 *   out[b,h,i,:] = sum_j softmax_j(scale * <q_i, k_j> | allowed(i,j)) v_j
 *   lse[b,h,i]   = ln sum_{j allowed} exp(scale * <q_i, k_j>)
 * q, k, v, out: [B, heads, N, d] of dtype; lse: float32 [B, heads, N] or NULL.
 * A query with no allowed key gets out = 0 and lse = -inf.
 * out may not alias q, k or v. The mask must have been built for this N.
 * bf16: products on bf16 matrix cores, fp32 accumulation and softmax, out
 * rounded to bf16. f32: fp32 arithmetic throughout.
 * Supported: d in {32, 64}; tile_m in {64, 128}; tile_n == 64 (any N: on a
 * ragged tiling only rows < N are read or written); otherwise UNSUPPORTED.
 */
hla_status hla_attn_fwd(const void *q, const void *k, const void *v,
                        const hla_block_mask *mask, void *out, float *lse,
                        int64_t B, int64_t heads, int64_t N, int64_t d,
                        hla_dtype dtype, float scale, hla_stream_t stream);

/*
 * The same attention forward with the reordering fused into its loads and
 * stores, so that no separate gather or scatter pass is needed (the paper's
 * "reshape" step, Sec. 4.2, done inside the attention instead of around it).
 * q, k, v, out are stored in grid order (row-major tokens); sequence position i
 * (the position the mask's pattern refers to) is row order[i]:
 *   out[b,h,order[i],:] = hla_attn_fwd's out[b,h,i,:] for
 *                         q'[b,h,i,:] = q[b,h,order[i],:] (likewise k', v'),
 *   lse[b,h,order[i]]   = the same row's lse.
 * The results equal hla_gather -> hla_attn_fwd -> hla_scatter bit for bit.
 * order: device int32[N], a permutation of [0, N) (not checked; an out-of-range
 * entry is undefined behaviour), 16-byte aligned, not overlapping any tensor
 * (typically hla_hilbert_perm's order). Other arguments, support and errors as
 * hla_attn_fwd.
 */
hla_status hla_attn_fwd_perm(const void *q, const void *k, const void *v,
                             const int32_t *order, const hla_block_mask *mask,
                             void *out, float *lse, int64_t B, int64_t heads,
                             int64_t N, int64_t d, hla_dtype dtype, float scale,
                             hla_stream_t stream);

/*
 * hla_attn_fwd_perm with the Hilbert index and the tile lists computed inside
 * the kernel, so that the whole step of a Hilbert attention - curve, tile lists,
 * reordered attention (Sec. 3.1-3.2; the reshape of Sec. 4.2 fused in) - is one
 * launch with no metadata in memory. Every workgroup takes its rows' grid ids
 * from the curve of the 2^k x 2^k grid (the order hla_hilbert_perm writes: 64
 * consecutive positions from a multiple of 64 are one aligned 8 x 8 block of the
 * curve) and classifies its row of tiles with hla_build_block_mask's classifier.
 * q, k, v, out: bf16 [B, heads, N, d] in grid order, as hla_attn_fwd_perm.
 * lse: as hla_attn_fwd_perm (may be NULL).
 * pat: a Hilbert pattern (window, slide, neighborhood, shifted window) on a grid
 * with H == W == 2^k >= 8; N must equal H * W. tile_m, tile_n, d: as
 * hla_attn_fwd (128 x 64 or 64 x 64; d 32 or 64). The results equal
 * hla_hilbert_perm -> hla_build_block_mask -> hla_attn_fwd_perm bit for bit.
 * A workgroup serves one query tile for up to 8 consecutive (batch, head)
 * slices, chosen by the library from the pattern's key span and the grid size;
 * the environment variable HLA_ATTN_HEADS_PER_WORKGROUP (1 .. 64) sets that
 * number instead (read at every call; the results do not depend on it).
 * Errors: HLA_ERR_UNSUPPORTED for other patterns, grids or dtypes (use
 * hla_attn_fwd_perm with a precomputed order and mask); otherwise as
 * hla_attn_fwd.
 */
hla_status hla_attn_fwd_hilbert(const void *q, const void *k, const void *v,
                                const hla_pattern_desc *pat, int32_t tile_m, int32_t tile_n,
                                void *out, float *lse, int64_t B, int64_t heads, int64_t N,
                                int64_t d, hla_dtype dtype, float scale, hla_stream_t stream);

/*
 * The attention forward with the global relative position bias of the Hilbert
 * Window Transformer (Sec. 3.2: the Swin window bias enlarged to the whole
 * feature map, because Hilbert windows have irregular shapes; Eq. 1 counts such
 * a score modification in the per-block work):
 *   S_ij = scale * <q_i, k_j> + rpb[h, r_i - r_j + H - 1, c_i - c_j + W - 1]
 * where (r_i, c_i) = (order[i] / W, order[i] % W) is the grid cell of sequence
 * position i, and H, W are the mask's grid. q, k, v, out, lse in sequence order
 * as for hla_attn_fwd.
 * order: device int32[N], the grid (row-major) id of each sequence position
 * (hla_hilbert_perm's order for the Hilbert patterns; 0, 1, ..., N-1 for the
 * row-major ones), 16-byte aligned, entries in [0, N) (not checked).
 * rpb: device float32 [heads, 2H-1, 2W-1], the same for every batch element.
 * Neither may overlap a tensor. Other arguments, support and errors as
 * hla_attn_fwd.
 */
hla_status hla_attn_fwd_rpb(const void *q, const void *k, const void *v,
                            const int32_t *order, const float *rpb,
                            const hla_block_mask *mask, void *out, float *lse,
                            int64_t B, int64_t heads, int64_t N, int64_t d,
                            hla_dtype dtype, float scale, hla_stream_t stream);

/*
 * Block-sparse attention backward: the gradients of hla_attn_fwd's out with
 * respect to q, k and v for an upstream gradient dout, over the same tiles as
 * the forward (empty tiles skipped, partial tiles masked; the paper times this
 * pass beside the forward for every pattern, Tables 1, 3, 6, 7, 9, 11). With the forward's lse:
 *   P[i,j]  = exp(scale * <q_i, k_j> - lse_i)  if allowed(i, j), else 0
 *   delta_i = <dout_i, out_i>                  (= sum_j P[i,j] <dout_i, v_j>)
 *   dS[i,j] = P[i,j] * (<dout_i, v_j> - delta_i)
 *   dq_i = scale * sum_j dS[i,j] k_j,   dk_j = scale * sum_i dS[i,j] q_i,
 *   dv_j = sum_i P[i,j] dout_i.
 * q, k, v, out, dout: [B, heads, N, d] of dtype, with out and lse exactly as
 * returned by hla_attn_fwd for these q, k, v, mask and scale.
 * lse: float32 [B, heads, N] (required).
 * stats: caller-owned float32 [B, heads, N, 2] workspace, overwritten with
 * (lse_i * log2(e), -delta_i) per row (+inf in place of the first where
 * lse_i = -inf).
 * dq, dk, dv: [B, heads, N, d] of dtype; they may not overlap each other or any
 * input. A query with no allowed key contributes nothing.
 * The mask must carry the transposed lists (see hla_block_mask).
 * Deterministic: every output element is written by exactly one thread, with a
 * fixed summation order (no atomics).
 * bf16: products on bf16 matrix cores with P and dS rounded to bf16 as
 * operands, fp32 accumulation, gradients rounded to bf16. f32: fp32 throughout.
 * With bf16 and tile_m == 128 a dk/dv workgroup may run its key tile for up
 * to 8 consecutive heads in turn (chosen from the GPU's size and the pattern;
 * the environment variable HLA_ATTN_BWD_HEADS_PER_WORKGROUP (1 .. 64) sets
 * that count, read at every call); the results do not depend on it. The same
 * holds for hla_attn_bwd_perm and hla_attn_bwd_noalloc.
 * Supported: d in {32, 64}; tile_m in {64, 128}; tile_n == 64;
 * otherwise UNSUPPORTED.
 */
hla_status hla_attn_bwd(const void *q, const void *k, const void *v, const void *out,
                        const void *dout, const float *lse, const hla_block_mask *mask,
                        void *dq, void *dk, void *dv, float *stats, int64_t B,
                        int64_t heads, int64_t N, int64_t d, hla_dtype dtype, float scale,
                        hla_stream_t stream);

/*
 * The same backward pass with the reordering fused into its loads and stores,
 * the counterpart of hla_attn_fwd_perm for training: q, k, v, out, dout, lse,
 * dq, dk, dv and stats are all stored in grid (row-major) order, and sequence
 * position i (the position the mask's pattern refers to) is row order[i]:
 *   dq[b,h,order[i],:] = hla_attn_bwd's dq[b,h,i,:] for the inputs taken in
 *   sequence order (q'[b,h,i,:] = q[b,h,order[i],:], likewise k, v, out, dout,
 *   lse), and the same for dk, dv.
 * out and lse are hla_attn_fwd_perm's results for these q, k, v, order, mask and
 * scale. order: device int32[N], a permutation of [0, N) (not checked),
 * 16-byte aligned, not overlapping an output or stats. The results equal
 * gather -> hla_attn_bwd -> scatter bit for bit. Other arguments, support and
 * errors as hla_attn_bwd.
 */
hla_status hla_attn_bwd_perm(const void *q, const void *k, const void *v, const void *out,
                             const void *dout, const float *lse, const int32_t *order,
                             const hla_block_mask *mask, void *dq, void *dk, void *dv,
                             float *stats, int64_t B, int64_t heads, int64_t N, int64_t d,
                             hla_dtype dtype, float scale, hla_stream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): hla_attn_bwd without
 * the stats workspace. The row statistics go instead to an array this library
 * holds on every device it runs on: 8 MiB (two floats for each of 2^20 rows),
 * held from the library's load on that device until the process ends. So
 * B * heads * N must be at most 1048576; a larger call returns
 * HLA_ERR_UNSUPPORTED (hla_attn_bwd takes any size).
 * The call allocates and frees nothing. It runs on the current device; stream,
 * if not NULL, must belong to it (else HLA_ERR_INVALID_ARG). Its first call on
 * a device looks the array's address up once (hipGetSymbolAddress).
 * Every call on one device shares that device's array, which keeps the last
 * call's contents. Calls in one stream's order are safe. Calls whose work
 * overlaps in time on one device (on different streams, or from several
 * threads) race on the array and give wrong gradients; serialise them. The
 * array needs no clearing: each call's first kernel writes the statistics of
 * every row before its second kernel reads them.
 * Results equal hla_attn_bwd's bit for bit. Other arguments, support and errors
 * as hla_attn_bwd.
 */
hla_status hla_attn_bwd_noalloc(const void *q, const void *k, const void *v, const void *out,
                                const void *dout, const float *lse, const hla_block_mask *mask,
                                void *dq, void *dk, void *dv, int64_t B, int64_t heads, int64_t N,
                                int64_t d, hla_dtype dtype, float scale, hla_stream_t stream);

/*
 * QKV projection with head split (Sec. 4.2, input processing: the Linear layer
 * that produces Q, K, V from the token features):
 *   y = x W_qkv^T,  x [B, N, C],  W_qkv [3C, C] (row f is output feature f),
 *   q[b,h,n,e] = y[b,n,      h*d + e]
 *   k[b,h,n,e] = y[b,n,  C + h*d + e]
 *   v[b,h,n,e] = y[b,n, 2C + h*d + e],   C = heads * d, no bias.
 * bf16 in and out, fp32 accumulation. q, k, v: [B, heads, N, d].
 * Supported: d == 32 or 64, C a multiple of 64; otherwise UNSUPPORTED.
 */
hla_status hla_qkv_proj(const void *x, const void *w_qkv, void *q, void *k,
                        void *v, int64_t B, int64_t N, int64_t heads, int64_t d,
                        hla_stream_t stream);

/*
 * Output projection with head merge:
 *   y[b,n,f] = sum_{h,e} o[b,h,n,e] * W_proj[f, h*d + e],  no bias.
 * o: [B, heads, N, d]; W_proj: [C_out, heads*d]; y: [B, N, C_out]; bf16, fp32
 * accumulation. Supported: d == 32 or 64, C_out a multiple of 64.
 */
hla_status hla_out_proj(const void *o, const void *w_proj, void *y, int64_t B,
                        int64_t N, int64_t heads, int64_t d, int64_t c_out,
                        hla_stream_t stream);

/*
 * The two projections with the token reordering fused in (the reshape step of
 * Sec. 4.2 done inside the projections' loads and stores), for a layer whose
 * features stay in grid (row-major) order while its attention runs in sequence
 * order: order is hla_hilbert_perm's order (sequence position n of the grid is
 * row order[n]).
 *   hla_qkv_proj_perm: x [B, N, C] in grid order; q, k, v in sequence order:
 *     q[b,h,n,:] = hla_qkv_proj's q for the input row x[b, order[n], :]
 *     (likewise k, v), i.e. gather -> hla_qkv_proj in one pass.
 *   hla_out_proj_perm: o in sequence order; y [B, N, C_out] in grid order:
 *     y[b, order[n], :] = hla_out_proj's y[b, n, :], i.e. hla_out_proj ->
 *     scatter in one pass.
 * order: device int32[N], a permutation of 0 .. N-1 (entries in [0, N), not
 * checked), 16-byte aligned, overlapping no output. The results equal the
 * composed calls bit for bit. Other arguments, support and errors as
 * hla_qkv_proj / hla_out_proj; a null order is INVALID_ARG.
 */
hla_status hla_qkv_proj_perm(const void *x, const void *w_qkv, const int32_t *order,
                             void *q, void *k, void *v, int64_t B, int64_t N,
                             int64_t heads, int64_t d, hla_stream_t stream);
hla_status hla_out_proj_perm(const void *o, const void *w_proj, const int32_t *order,
                             void *y, int64_t B, int64_t N, int64_t heads, int64_t d,
                             int64_t c_out, hla_stream_t stream);

/* Text of the last non-OK status returned on this thread ("" if none). */
const char *hla_last_error(void);

/* Library version string. */
const char *hla_version(void);

#ifdef __cplusplus
}
#endif

#endif /* HLA_H */
