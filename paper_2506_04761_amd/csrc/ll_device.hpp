// Device-side building blocks shared by the libloglinear kernels (gfx950 / CDNA4).
//
//  * MFMA traits: one 16x16 output tile per instruction, bf16 (16x16x32) or fp32 (16x16x4).
//    Operand convention used everywhere: lane l supplies row (A) or column (B) l & 15, and the
//    KPL consecutive k values starting at (l >> 4) * KPL of the current k step.  A contraction
//    only needs A and B to agree on which k each (lane group, slot) carries, so the same
//    convention serves every operand loaded from memory.  The 16x16 fp32 result tile is held
//    as lane l: column l & 15, rows 4 * (l >> 4) + r for r = 0..3.
//  * Fenwick level functions (Sec. 3.1 footnote): l(t, s) = bit length of t XOR s for s <= t,
//    and the source group a block of tokens reads at each level above it (Sec. 3.3, Eq. 5).
//  * A wave-wide inclusive prefix sum for the block-local cumulative log-gates (Eq. 2).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ll {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;

// 2^x with the hardware v_exp_f32 (arguments here are always <= 0; results below the normal
// range may flush to zero, which only drops terms already negligible against the others).
__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <typename T>
struct Mfma;

template <>
struct Mfma<__bf16> {
  static constexpr int KSTEP = 32;  // k per instruction
  static constexpr int KPL = 8;     // k values per lane
  typedef bf16x8 frag;
  __device__ static inline f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static inline frag load(const __bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }
};

template <>
struct Mfma<float> {
  static constexpr int KSTEP = 4;
  static constexpr int KPL = 1;
  typedef float frag;
  __device__ static inline f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  __device__ static inline frag load(const float* p) { return *p; }
};

// Transposing LDS read (ds_read_b64_tr_b16, gfx950).  Within each group of 16 lanes, lane j
// supplies the address of four consecutive 16-bit elements e_j[0..3]; lane i receives
// { e_(i/4 + 4k)[i % 4] : k = 0..3 }.  Supplying, from lane j of the group, row (base + j/4)
// and column (c0 + 4 (j % 4)) of a row-major matrix therefore hands lane i column c0 + i of
// rows base .. base + 3: a 4 x 16 block read as 16 columns, i.e. an MFMA operand fragment whose
// k slots run down the rows.
__device__ inline bf16x4 lds_read_tr(const __bf16* p) {
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  const s16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
  return __builtin_bit_cast(bf16x4, r);
}

// bf16 MFMA operand fragment (8 k slots) taken down the rows of a row-major bf16 matrix in LDS:
// lane (g = lane / 16, i = lane % 16) gets column col0 + i at rows row0 + 4g + {0..3} (slots
// 0-3) and row0 + 16 + 4g + {0..3} (slots 4-7).  `ld` is the row stride in elements.
__device__ inline bf16x8 frag_down_rows(const __bf16* m, int ld, int row0, int col0) {
  const int lane = threadIdx.x & 63, g = lane >> 4, i = lane & 15;
  const __bf16* p = m + (row0 + 4 * g + (i >> 2)) * ld + col0 + 4 * (i & 3);
  const bf16x4 lo = lds_read_tr(p);
  const bf16x4 hi = lds_read_tr(p + 16 * ld);
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// 16-byte vector of storage elements, for coalesced global <-> LDS copies.
template <typename T>
struct Vec16 {
  static constexpr int N = 16 / sizeof(T);
  typedef T type __attribute__((ext_vector_type(16 / sizeof(T))));
};

__device__ inline float to_f32(float x) { return x; }
__device__ inline float to_f32(__bf16 x) { return static_cast<float>(x); }
template <typename T>
__device__ inline T from_f32(float x) { return static_cast<T>(x); }

// ----------------------------------------------------------------------------------- levels

// Bit length of x (0 for x == 0).
__device__ __host__ inline int bitlen(uint32_t x) { return x ? 32 - __builtin_clz(x) : 0; }

// Level of key position s seen from query position t, both inside one power-of-two-aligned
// block of P tokens and given as block-local indices (i = t mod P, j = s mod P, j <= i).
// Because the block start is a multiple of P, the global XOR equals the local one.
__device__ __host__ inline int level_local(int i, int j) { return bitlen(uint32_t(i ^ j)); }

// Source group (Sec. 3.3, Eq. 5), for aligned blocks of P = 2^p tokens (chunks in the paper,
// tiles of two chunks here): block z reads a term at block level j >= 1 (token level p + j) iff
// bit j-1 of z is set; the keys then come from the block range [first, first + 2^(j-1)) with
// first = ((z >> (j-1)) - 1) << (j-1), the 2^(j-1) blocks immediately before z's own aligned
// 2^(j-1)-block.
__device__ __host__ inline bool reads_level(int64_t z, int j) { return (z >> (j - 1)) & 1; }
__device__ __host__ inline int64_t source_first(int64_t z, int j) { return ((z >> (j - 1)) - 1) << (j - 1); }
// The same group by its end: the level-j group of block z (bit j - 1 of z set) is the 2^(j-1)
// blocks before group_end(z, j); group_end has exactly j - 1 trailing zeros.
__device__ __host__ inline int64_t group_end(int64_t z, int j) { return (z >> (j - 1)) << (j - 1); }

// level_local(i, j) of a 128-row tile as the 16 x 16 MFMA tiles see it (i = 16 gi + r,
// j = 16 gj + c): inside one 16-row group the level is that of the in-group indices; across groups
// (gj < gi) it is 4 + the level of the group indices, one level for the whole 16 x 16 tile.
__device__ __host__ inline int level_in_group(int r, int c) { return bitlen(uint32_t(r ^ c)); }
__device__ __host__ inline int level_across_groups(int gi, int gj) { return 4 + bitlen(uint32_t(gi ^ gj)); }

// ------------------------------------------------------------------ direct global -> LDS tiles
//
// Row-major bf16 tiles whose 16-byte chunks are XOR-swizzled by row (chunk c of row r sits at
// position c ^ (r mod chunks-per-row)), filled by direct global->LDS loads
// (global_load_lds_dwordx4: lane l of a wave instruction writes bytes 16 l .. 16 l + 15 of a
// 1 KiB span).  A fragment read down 16 consecutive rows then touches 16 different positions.

// Element offset of 16-byte chunk c of row r in a swizzled row-major bf16 tile of D columns.
template <int D>
__device__ inline int swz(int r, int c) {
  return r * D + ((c ^ (r & (D / 8 - 1))) << 3);
}

// Copies ROWS rows of D bf16 elements (row r at src + r * stride) into the swizzled LDS tile
// `dst` by direct global->LDS loads, one 1 KiB span per wave instruction, spans dealt to the NT/64
// waves in turn.  Rows at or beyond `nrow` are filled from row nrow - 1 (callers never read
// them).  The copy is complete once the issuing wave has waited for its vector-memory operations.
// AUX: cache-policy bits of the loads (0 by default; 2, non-temporal, for data read once).
template <int D, int ROWS, int NT, int AUX = 0>
__device__ inline void lds_copy_rows(__bf16* dst, const __bf16* __restrict__ src, int64_t stride, int nrow) {
  constexpr int CH = D / 8;      // chunks per row
  constexpr int RPI = NT / CH;   // rows per pass of all waves
  static_assert(NT % CH == 0 && RPI % CH == 0 && ROWS % RPI == 0, "whole rows per pass");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int q0 = wave * 64 + lane;                     // chunk position in the first pass
  const int r0 = q0 / CH, c = (q0 % CH) ^ (r0 & (CH - 1));  // the swizzle repeats every pass
#pragma unroll
  for (int it = 0; it < ROWS / RPI; ++it) {
    const int r = r0 + it * RPI;
    const int rs = r < nrow ? r : nrow - 1;
    __builtin_amdgcn_global_load_lds(src + rs * stride + c * 8,
                                     (__attribute__((address_space(3))) void*)(dst + (it * NT + wave * 64) * 8), 16, 0,
                                     AUX);
  }
}

// bf16 MFMA operand fragment down the rows of a swizzled tile (as frag_down_rows).
template <int D>
__device__ inline bf16x8 frag_down_rows_swz(const __bf16* m, int row0, int col0) {
  const int lane = threadIdx.x & 63, g = lane >> 4, i = lane & 15;
  const int r = row0 + 4 * g + (i >> 2), col = col0 + 4 * (i & 3);
  const bf16x4 lo = lds_read_tr(m + swz<D>(r, col >> 3) + (col & 7));
  const bf16x4 hi = lds_read_tr(m + swz<D>(r + 16, col >> 3) + (col & 7));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// bf16 MFMA operand fragment along a row of a swizzled tile: row row0 + (lane % 16), the 8
// elements starting at column 8 * chunk0 + 8 * (lane / 16).
template <int D>
__device__ inline bf16x8 frag_along_row_swz(const __bf16* m, int row0, int chunk0) {
  const int lane = threadIdx.x & 63;
  return *reinterpret_cast<const bf16x8*>(m + swz<D>(row0 + (lane & 15), chunk0 + (lane >> 4)));
}

// Copies n 16-byte pieces (n a multiple of 64) into LDS, piece q to dst + 16 q bytes, from global
// addresses src(q), by direct global->LDS loads; the NT/64 waves take 64 pieces in turn.
template <int NT, typename Src>
__device__ inline void lds_gather16(void* dst, int n, Src src) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (int s0 = wave * 64; s0 < n; s0 += NT)
    __builtin_amdgcn_global_load_lds(src(s0 + lane),
                                     (__attribute__((address_space(3))) void*)((char*)dst + s0 * 16), 16, 0, 0);
}

// As lds_gather16 for 4-byte pieces: piece q to dst + 4 q bytes.
template <int NT, typename Src>
__device__ inline void lds_gather4(void* dst, int n, Src src) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  for (int s0 = wave * 64; s0 < n; s0 += NT)
    __builtin_amdgcn_global_load_lds(src(s0 + lane),
                                     (__attribute__((address_space(3))) void*)((char*)dst + s0 * 4), 4, 0, 0);
}

// Waits for this wave's outstanding vector-memory operations (including direct-to-LDS loads).
__device__ inline void wait_vmem() { __builtin_amdgcn_s_waitcnt(0); }

// Waits until at most N of this wave's vector-memory operations are outstanding (they complete in
// issue order); memory accesses are not moved across it.
template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// ------------------------------------------------------------------------- dispatch order

// MI355X has 8 XCDs, each with its own L2, and hands out workgroups round-robin over them.
// Remapping the dispatch index this way gives each XCD one contiguous range of logical work
// items, so neighbours in logical order (the two halves of a tile, consecutive tiles of one
// head that share summaries) run on the same XCD and share its L2.
constexpr int kXcds = 8;
__device__ inline int64_t xcd_remap(int64_t id, int64_t total) {
  const int64_t q = total / kXcds, rem = total % kXcds;
  const int64_t xcd = id % kXcds, slot = id / kXcds;
  return xcd * q + (xcd < rem ? xcd : rem) + slot;
}

// ----------------------------------------------------------------------------- wave helpers

// Inclusive prefix sum across the 64 lanes of a wave (Hillis-Steele over DPP/permute).
__device__ inline float wave_inclusive_scan(float x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    float y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  return x;
}

}  // namespace ll
