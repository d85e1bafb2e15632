// Device helpers shared by the attention kernels (forward and backward, bf16 and
// fp32): the allowed region of a position under a pattern, the element mask over
// an MFMA accumulator, the gfx950 LDS primitives, and the grid remap.
#pragma once

#include "hla_internal.h"

namespace hla {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

__device__ __forceinline__ int clampi(int x, int lo, int hi) { return min(max(x, lo), hi); }

// Workgroups are dealt round-robin to the 8 XCDs; remap so that each XCD gets a
// contiguous range of logical tiles (neighbouring tiles share key / value or
// query tiles, and the reuse then stays in one XCD's L2).
__device__ __forceinline__ int xcd_remap(int bid, int total) {
  const int per = total >> 3, rem = total & 7;
  const int xcd = bid & 7, slot = bid >> 3;
  return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

// Scalar (SMEM) load of a wave-uniform int through the constant address space.
__device__ __forceinline__ int sload(const int32_t *p) {
  return *(const __attribute__((address_space(4))) int32_t *)p;
}

// ---------------------------------------------------------------------------
// Allowed regions (Sec. 3.1-3.3). For a fixed position x the positions it pairs
// with form one interval [lo, hi] for the 1-D (Hilbert-sequence) patterns and one
// rectangle of grid cells [rlo, rhi] x [clo, chi] for the row-major patterns.
// region_of<true>(P, x): the keys query x may attend. region_of<false>(P, x):
// the queries that may attend key x (the same relation read the other way; only
// the neighbourhood patterns are not symmetric).

// (The row-major patterns keep their row range [rlo, rhi] in lo, hi.)
struct Region {
  bool one_d;
  int lo, hi, clo, chi;
};

// Neighbourhood of length k on an axis of `extent` cells: query x attends
// [s(x), s(x) + k) with s(x) = clamp(x - k/2, 0, extent - k).
__device__ __forceinline__ void neigh_fwd(int x, int k, int extent, int &lo, int &hi) {
  lo = clampi(x - k / 2, 0, extent - k);
  hi = lo + k - 1;
}
// Queries x with s(x) <= y < s(x) + k. s is non-decreasing, so they form an
// interval: s(x) <= y holds for all x if y >= extent - k, else for x <= y + k/2;
// s(x) >= y - k + 1 holds for all x if y - k + 1 <= 0, else for x >= y - k + 1 + k/2.
__device__ __forceinline__ void neigh_bwd(int y, int k, int extent, int &lo, int &hi) {
  hi = y >= extent - k ? extent - 1 : y + k / 2;
  lo = y - k + 1 <= 0 ? 0 : y - k + 1 + k / 2;
}

template <bool KEYS_OF_QUERY>
__device__ __forceinline__ Region region_of(const PatternArgs &P, int x) {
  Region R;
  R.one_d = P.kind == HLA_HILBERT_WINDOW || P.kind == HLA_HILBERT_SLIDE ||
            P.kind == HLA_HILBERT_NEIGHBORHOOD || P.kind == HLA_HILBERT_SHIFTED_WINDOW;
  R.lo = R.hi = R.clo = R.chi = 0;
  if (P.kind == HLA_HILBERT_WINDOW) {
    R.lo = (x / P.p0) * P.p0;
    R.hi = R.lo + P.p0 - 1;
  } else if (P.kind == HLA_HILBERT_SLIDE) {
    R.lo = x - P.p0;
    R.hi = x + P.p0;
  } else if (P.kind == HLA_HILBERT_NEIGHBORHOOD) {
    if (KEYS_OF_QUERY) neigh_fwd(x, P.p0, P.N, R.lo, R.hi);
    else neigh_bwd(x, P.p0, P.N, R.lo, R.hi);
  } else if (P.kind == HLA_HILBERT_SHIFTED_WINDOW) {
    const int g = (x + P.p0 - P.p1) / P.p0;
    R.lo = g * P.p0 - P.p0 + P.p1;
    R.hi = R.lo + P.p0 - 1;
  } else {
    const int r = (int)fdiv((uint32_t)x, P.wdiv), c = x - r * P.W;
    if (P.kind == HLA_ROWMAJOR_WINDOW) {
      R.lo = (r / P.p0) * P.p0; R.hi = R.lo + P.p0 - 1;
      R.clo = (c / P.p1) * P.p1; R.chi = R.clo + P.p1 - 1;
    } else if (P.kind == HLA_ROWMAJOR_SLIDE) {
      R.lo = r - P.p0; R.hi = r + P.p0;
      R.clo = c - P.p1; R.chi = c + P.p1;
    } else if (KEYS_OF_QUERY) {
      neigh_fwd(r, P.p0, P.H, R.lo, R.hi);
      neigh_fwd(c, P.p1, P.W, R.clo, R.chi);
    } else {
      neigh_bwd(r, P.p0, P.H, R.lo, R.hi);
      neigh_bwd(c, P.p1, P.W, R.clo, R.chi);
    }
  }
  // Clip at the end of the sequence: on a ragged tiling the edge tiles hold
  // padded positions >= N (grid rows >= H), which pair with nothing.
  R.hi = min(R.hi, R.one_d ? P.N - 1 : P.H - 1);
  return R;
}

__device__ __forceinline__ bool region_has(const Region &R, const PatternArgs &P, int y) {
  if (R.one_d) return y >= R.lo && y <= R.hi;
  const int r = (int)fdiv((uint32_t)y, P.wdiv), c = y - r * P.W;
  return r >= R.lo && r <= R.hi && c >= R.clo && c <= R.chi;
}

// Element mask over NB 32x32 accumulator blocks. Slot v of this lane in block
// kb holds the position base + 32*kb + 16*(v/8) + v%8 (runs of eight
// consecutive positions; base = first position of block 0 + 8 * lane half).
// Disallowed entries become -inf. For the row-major patterns with W a multiple
// of 8 a run never crosses a grid row, so one division per run. The pattern
// branch is taken once for all blocks.
//
// 1-D patterns: the lane's allowed slots are the offsets c = position - base in
// [R.lo - base, R.hi - base]. A partial tile at the edge of a band or a window
// usually cuts that interval on one side only, for every lane of the wave; two
// ballots find out, and then one compare per entry against the cut side's bound
// does (instead of the two-sided unsigned compare, which needs an add per
// entry), or nothing at all when no lane of the wave loses a slot. (A row with
// an empty interval - only padded rows past the end of the sequence, whose
// results are never stored - may keep slots; every stored row is exact.)
template <int NB>
__device__ __forceinline__ void mask_blocks(f32x16 (&s)[NB], const Region &R,
                                            const PatternArgs &P, int base) {
  if (R.one_d) {
    constexpr int CMAX = 32 * (NB - 1) + 23;   // largest offset a lane holds
    const int lo = R.lo - base, hi = R.hi - base;
    const bool cut_lo = __ballot(lo > 0) != 0;
    const bool cut_hi = __ballot(hi < CMAX) != 0;
    if (!cut_lo && !cut_hi) return;
    if (cut_lo && cut_hi) {
      const uint32_t span = (uint32_t)(hi - lo);
#pragma unroll
      for (int kb = 0; kb < NB; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const bool ok = (uint32_t)(32 * kb + 16 * (v >> 3) + (v & 7) - lo) <= span;
          s[kb][v] = ok ? s[kb][v] : -__builtin_inff();
        }
    } else if (cut_lo) {   // every lane keeps all slots from its lower bound on
#pragma unroll
      for (int kb = 0; kb < NB; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          s[kb][v] = 32 * kb + 16 * (v >> 3) + (v & 7) >= lo ? s[kb][v] : -__builtin_inff();
    } else {               // every lane keeps all slots up to its upper bound
#pragma unroll
      for (int kb = 0; kb < NB; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          s[kb][v] = 32 * kb + 16 * (v >> 3) + (v & 7) <= hi ? s[kb][v] : -__builtin_inff();
    }
  } else if ((P.W & 7) == 0) {
    const uint32_t rspan = (uint32_t)(R.hi - R.lo), cspan = (uint32_t)(R.chi - R.clo);
#pragma unroll
    for (int kb = 0; kb < NB; ++kb)
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const int y0 = base + 32 * kb + 16 * g;
        const int r = (int)fdiv((uint32_t)y0, P.wdiv);
        const int c0 = y0 - r * P.W - R.clo;
        const bool row_ok = (uint32_t)(r - R.lo) <= rspan;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const bool ok = row_ok & ((uint32_t)(c0 + t) <= cspan);
          s[kb][8 * g + t] = ok ? s[kb][8 * g + t] : -__builtin_inff();
        }
      }
  } else {
#pragma unroll
    for (int kb = 0; kb < NB; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const bool ok = region_has(R, P, base + 32 * kb + 16 * (v >> 3) + (v & 7));
        s[kb][v] = ok ? s[kb][v] : -__builtin_inff();
      }
  }
}

// ---------------------------------------------------------------------------
// MFMA operand layout helpers (v_mfma_f32_32x32x16_bf16).
//
// The accumulator of a 32x32 MFMA holds, in lane (col = l%32, half = l/32) and
// slot v, row 8*(v/4) + 4*half + v%4. Feeding the A operand's rows permuted by
// row_perm makes slot v of lane half `half` hold row 16*(v/8) + 8*half + v%8:
// runs of eight consecutive rows, which is exactly the B-operand layout of a
// second MFMA that contracts over those rows in 16-row steps (slots 8t..8t+7 are
// the lane's operand for step t). So a product's result feeds the next product
// from registers, with no LDS round trip.
__device__ __forceinline__ int row_perm(int i) {
  // accumulator row i = 8a + 4g + b  ->  operand row 16(a/2) + 8g + 4(a%2) + b
  const int a = i >> 3, g = (i >> 2) & 1, b = i & 3;
  return 16 * (a >> 1) + 8 * g + 4 * (a & 1) + b;
}

// LDS byte address of a pointer into __shared__ memory.
__device__ __forceinline__ uint32_t lds_addr(const void *p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char *)p;
}

// ---------------------------------------------------------------------------
// gfx950 LDS DMA (16 bytes per lane; lane l lands at dst + 16 l), issued from
// inline assembly (M0 = the wave's LDS destination, then the load), and the
// transposing 64-bit LDS read. Only the device pass may see these: the host
// pass of the HIP compiler rejects the builtins silently and then emits no
// launch stub for the kernel that calls them.
//
// The compiler cannot see this copy, so it inserts no wait of
// its own for it: a kernel that uses it must order every LDS read of the copied
// data after the copy itself - an explicit vmcnt wait for the wave's own copies
// followed by a workgroup barrier. In exchange the compiler's wait insertion no
// longer treats later LDS reads as possibly overlapping a copy in flight (for
// the transposing read below it would otherwise wait for every outstanding
// copy, draining a copy ring on every tile). dst must be wave-uniform.
// M0 is a reserved register, so the compiler does not preserve a value of its
// own across this statement; nothing else in these kernels uses M0 (the
// compiler's own LDS DMA builtin would, which is why it is not used here).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_dma16(const void *src, uint32_t dst) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(__builtin_amdgcn_readfirstlane(dst))
               : "memory", "m0");
#endif
}
// The same copy from a wave-uniform base plus a per-lane 32-bit byte offset (the
// saddr form): the 64-bit address add happens in the memory pipeline instead of
// taking two vector instructions per copy. The offset must stay below 2^31.
__device__ __forceinline__ void lds_dma16_at(const void *base, uint32_t off, uint32_t dst) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(off), "s"(base), "s"(__builtin_amdgcn_readfirstlane(dst))
               : "memory", "m0");
#endif
}
// The same copy with 4 bytes per lane (lane l lands at dst + 4 l; lanes that are
// switched off write nothing): row indices, where each lane clamps its own source
// position at the end of the sequence.
__device__ __forceinline__ void lds_dma4(const void *src, uint32_t dst) {
#if defined(__HIP_DEVICE_COMPILE__)
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :
               : "v"(src), "s"(__builtin_amdgcn_readfirstlane(dst))
               : "memory", "m0");
#endif
}
#pragma clang diagnostic pop
__device__ __forceinline__ i16x4 lds_read_tr16(const char *p) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)p);
#else
  return i16x4{};
#endif
}
// Two transposing reads four rows apart, as one 8-element bf16 operand.
__device__ __forceinline__ bf16x8 lds_read_tr16x2(const char *p, int row_bytes) {
  const i16x4 lo4 = lds_read_tr16(p);
  const i16x4 hi4 = lds_read_tr16(p + 4 * row_bytes);
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo4, hi4, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Wait for every vector memory operation of this wave, as an instruction the
// compiler's own wait insertion sees (it then knows its loads have landed). The
// empty statement in front keeps the compiler from scheduling loads written
// before this call after the wait.
__device__ __forceinline__ void wait_vmem_all() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0); expcnt, lgkmcnt unconstrained
}

// Wait until this wave's LDS reads are done and at most N of its vector memory
// operations (tile copies) are in flight, then barrier the workgroup. One asm
// statement with a memory clobber, so the compiler moves no memory access across
// it (a fence would instead wait for every copy in flight).
template <int N>
__device__ __forceinline__ void wait_then_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt out of range");
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}
// Wait until at most n of this wave's vector memory operations are in flight
// (0 <= n <= MAXN; a larger n waits for MAXN), then barrier the workgroup.
template <int MAXN>
__device__ __forceinline__ void wait_n_then_barrier(int n) {
  if constexpr (MAXN > 0) {
    if (n >= MAXN) {
      wait_then_barrier<MAXN>();
      return;
    }
    wait_n_then_barrier<MAXN - 1>(n);
  } else {
    wait_then_barrier<0>();
  }
}

// Dispatch on the number of tiles still allowed in flight (0 .. MAXA), LPT
// vector memory operations per tile.
template <int LPT, int MAXA>
__device__ __forceinline__ void wait_tiles_then_barrier(int after) {
  if constexpr (MAXA > 0) {
    if (after >= MAXA) {
      wait_then_barrier<MAXA * LPT>();
      return;
    }
    wait_tiles_then_barrier<LPT, MAXA - 1>(after);
  } else {
    wait_then_barrier<0>();
  }
}

}  // namespace hla
