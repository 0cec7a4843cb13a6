// Pieces shared by the log-linear Mamba-2 forward (ll_mamba2.hip) and backward
// (ll_mamba2_bwd.hip) kernels: tile geometry, the device view of the forward's level summaries,
// the decay gaps of a tile's levels, tile-local cumulative gates and register row staging.
#pragma once

#include "ll_device.hpp"
#include "ll_launch.hpp"

namespace ll {

// Tile rows R: two chunks (C >= 32), at least 64 tokens.  Levels up to log2 R are computed densely
// inside a tile, the ones above from summaries of whole tiles.
__host__ __device__ constexpr int tile_rows(int C) { return 2 * C >= 64 ? 2 * C : 64; }
constexpr int kBlockTiles = 4;    // tiles per block_state workgroup
constexpr int kKB = 64;           // keys staged in LDS at a time
constexpr int kMaxLevels = 24;    // Fenwick levels handled (T <= 2^23)

// Device view of the summaries (all in the storage dtype, layout [p][n] = d_v x d_k) and of their
// summed log2-gates.  Above the blocks, node (l, k) of the block tree (l >= 1) covers blocks
// [k 2^l, (k + 1) 2^l), i.e. the tiles of the level-(l + 3) source group with index k.
// Offset of level b in a (b, h) row of the single-pass forward's block sums (level b: the sums of
// the aligned blocks of 2^b tiles' log2-gates).
__device__ __host__ inline int64_t bsum_offset(int64_t N, int b) {
  int64_t off = 0;
  for (int x = 0; x < b; ++x) off += (N + (int64_t(1) << x) - 1) >> x;
  return off;
}

template <typename T>
struct Nodes {
  T* lvl1;         // [BH][ceil(N/2)]  tile states of even tiles
  T* lvl2;         // [BH][ceil(N/4)]  pair summaries of tiles 4b, 4b+1
  T* blocks;       // [BH][NB]         block summaries (4 tiles)
  T* upper;        // [BH][nup]        block-tree nodes of levels >= 1 (tile levels >= 4)
  const float* t1; // [BH][N]          tile totals (the level-1 source groups are single tiles)
  float* t2;       // [BH][ceil(N/4)]  totals of the pairs in lvl2
  float* t3;       // [BH][NB]         block totals
  float* tup;      // [BH][nup]        totals of the upper nodes
  float* cl;       // [BH][N][R]       tile-local inclusive cumulative log2-gates (rows past T repeat the last)
  int64_t n1, n2, nb, nup;  // per-(b,h) slot counts
  // Left by the single-pass forward instead (by_u non-null): the summary of the aligned group of
  // tiles ending at tile u in slot [b h][u] of by_u (d_v x d_k), the groups' totals in the block
  // sums `bsum` (rows of `bstride` floats).
  T* by_u;
  const float* bsum;
  int64_t bstride;
  // Slot of block-tree node (l >= 1, k): tree levels 1 .. l-1 come first, ceil(nb / 2^l') slots each.
  __device__ __host__ int64_t up_slot(int64_t bh, int l, int64_t k) const {
    int64_t off = 0;
    for (int ll = 1; ll < l; ++ll) off += (nb + (int64_t(1) << ll) - 1) >> ll;
    return bh * nup + off + k;
  }
  // Summary of the level-j source group that starts at tile f (f a multiple of 2^(j-1)).
  __device__ __host__ T* at(int64_t bh, int64_t N, int j, int64_t f, int SZ) const {
    if (by_u) return by_u + (bh * N + f + (int64_t(1) << (j - 1)) - 1) * SZ;
    if (j == 1) return lvl1 + (bh * n1 + (f >> 1)) * SZ;
    if (j == 2) return lvl2 + (bh * n2 + (f >> 2)) * SZ;
    if (j == 3) return blocks + (bh * nb + (f >> 2)) * SZ;
    return upper + up_slot(bh, j - 3, f >> (j - 1)) * SZ;
  }
  // Summed log2-gate of the same group.
  __device__ __host__ float tot(int64_t bh, int64_t N, int j, int64_t f) const {
    if (by_u) return bsum[bh * bstride + bsum_offset(N, j - 1) + (f >> (j - 1))];
    if (j == 1) return t1[bh * N + f];
    if (j == 2) return t2[bh * n2 + (f >> 2)];
    if (j == 3) return t3[bh * nb + (f >> 2)];
    return tup[up_slot(bh, j - 3, f >> (j - 1))];
  }
};

// Whether block-tree node (l, k) is read: as the level-(l + 3) source group, by the tiles of the
// next aligned group, when k is even and that group has a tile.  A read node covers whole blocks.
__device__ __host__ inline bool tree_node_read(int l, int64_t k, int64_t N) {
  return !(k & 1) && ((k + 1) << (l + 2)) < N;
}

// Log2-decay gaps of tile u's levels, lane j - 1 holding gap_j: the summed log2-gates of the
// tiles between the end of level j's source group and u.  Those tiles are exactly the source
// groups of u's lower set bits, so gap_j is the sum of their totals (an exclusive wave scan).
template <typename T>
__device__ inline float level_gaps(const Nodes<T>& nodes, int64_t bh, int64_t N, int64_t u, int J) {
  const int j = (threadIdx.x & 63) + 1;
  float t = 0.f;
  if (j <= J && reads_level(u, j)) t = nodes.tot(bh, N, j, source_first(u, j));
  return wave_inclusive_scan(t) - t;
}

// gap_j from the lane-per-level values of level_gaps (j uniform across the wave)
__device__ inline float gap_of(float gapv, int j) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gapv), j - 1));
}

// Tile-local inclusive cumulative sum of log2 gates for the R rows of a tile (rows >= nrow get
// a zero gate), computed by the first 4 waves of the workgroup (R/4 <= 64 rows each) into cl_s[R].
//
// tile_gate issues this thread's load of the raw log-gate (always from a valid address); the
// scaling to log2 and the masking of rows outside the tile happen in tile_cumsum_of, where the
// value is first needed, so that issuing the load never makes the wave wait for it.
template <int R>
__device__ inline float tile_gate(const float* __restrict__ log_alpha, int64_t row0, int nrow, int H, int h) {
  constexpr int RPW = R / 4;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = wave * RPW + lane;
  const int rs = (wave < 4 && lane < RPW && r < nrow) ? r : 0;
  return log_alpha[(row0 + rs) * H + h];
}

// Scan of the raw gates returned by tile_gate for a tile of nrow rows.  Starts and ends with a
// barrier.
template <int R>
__device__ inline void tile_cumsum_of(float la_raw, int nrow, float* cl_s, float* wsum_s) {
  constexpr int RPW = R / 4;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = wave * RPW + lane;
  const bool mine = wave < 4 && lane < RPW;  // waves beyond the first four only take the barriers
  const float la = (mine && r < nrow) ? la_raw * kLog2e : 0.f;
  float cl = wave_inclusive_scan(la);
  __syncthreads();
  if (wave < 4 && lane == 63) wsum_s[wave] = cl;
  __syncthreads();
  float base = 0.f;
  for (int w = 0; w < wave && w < 4; ++w) base += wsum_s[w];
  if (mine) cl_s[r] = base + cl;
  __syncthreads();
}

template <int R>
__device__ inline void tile_cumsum(const float* __restrict__ log_alpha, int64_t row0, int nrow, int H, int h,
                                   float* cl_s, float* wsum_s) {
  tile_cumsum_of<R>(tile_gate<R>(log_alpha, row0, nrow, H, h), nrow, cl_s, wsum_s);
}

// Register staging of one 64-row block of a [rows, H, D] tensor, loaded with 16-byte vectors by
// the NT threads of the workgroup (thread unit = one row's 16-byte column group, consecutive
// threads along the row); rows at or beyond `nrow` repeat row nrow - 1 (callers give them zero
// weight).  D is the width loaded
// (elements per row) and LDROW the row length of the tensor in memory.  Stored row-major.
template <typename T, int D, int NT, int LDROW = D>
struct RowBlock {
  static constexpr int VEC = Vec16<T>::N;
  static constexpr int PER_ROW = D / VEC;
  static constexpr int TOTAL = kKB * PER_ROW;
  static constexpr int LOADS = (TOTAL + NT - 1) / NT;
  typename Vec16<T>::type x[LOADS];
  __device__ inline void load(const T* __restrict__ src, int64_t row0, int r0, int nrow, int H, int h) {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int idx = threadIdx.x + NT * i;
      const int t = idx / PER_ROW, d0 = (idx % PER_ROW) * VEC;
      // rows at or beyond nrow repeat row nrow - 1 (no branch: the number of loads in flight
      // stays the same on every path)
      const int rr = r0 + t < nrow ? r0 + t : nrow - 1;
      if (TOTAL % NT == 0 || idx < TOTAL)
        x[i] = *reinterpret_cast<const typename Vec16<T>::type*>(src + ((row0 + rr) * H + h) * LDROW + d0);
      else
        x[i] = typename Vec16<T>::type{};
    }
  }
  __device__ inline void store_rows(T* dst, int ld) const {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int idx = threadIdx.x + NT * i;
      const int t = idx / PER_ROW, d0 = (idx % PER_ROW) * VEC;
      if (idx < TOTAL) *reinterpret_cast<typename Vec16<T>::type*>(&dst[t * ld + d0]) = x[i];
    }
  }
  // row-major copy with a per-row scale: dst[t * ld + d] = x[t][d] * scale[t]
  __device__ inline void store_rows_scaled(T* dst, int ld, const float* scale) const {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int idx = threadIdx.x + NT * i;
      const int t = idx / PER_ROW, d0 = (idx % PER_ROW) * VEC;
      if (idx >= TOTAL) continue;
      const float sc = scale[t];
      typename Vec16<T>::type y;
#pragma unroll
      for (int e = 0; e < VEC; ++e) y[e] = from_f32<T>(to_f32(x[i][e]) * sc);
      *reinterpret_cast<typename Vec16<T>::type*>(&dst[t * ld + d0]) = y;
    }
  }
};

// Copies lambda of the tile's rows into dst[r * kMaxLevels + l] (l < L; the other slots receive
// copies of valid entries and are never read) by direct global->LDS loads of one float per lane.
template <int ROWS, int NT, int AUX = 0>
__device__ inline void lds_copy_lambda(float* dst, const float* __restrict__ lam, int64_t row0, int H, int h, int L,
                                       int nrow) {
  constexpr int TOTAL = ROWS * kMaxLevels;
  static_assert(TOTAL % NT == 0, "whole passes");
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
  for (int it = 0; it < TOTAL / NT; ++it) {
    const int pos = it * NT + wave * 64 + lane;
    const int r = pos / kMaxLevels, l = pos % kMaxLevels;
    const int rs = r < nrow ? r : nrow - 1, ls = l < L ? l : L - 1;
    __builtin_amdgcn_global_load_lds(lam + ((row0 + rs) * H + h) * L + ls,
                                     (__attribute__((address_space(3))) void*)(dst + it * NT + wave * 64), 4, 0, AUX);
  }
}

int tile_levels(int64_t T, int64_t C);

// Device view of the summaries in a forward workspace laid out by mamba2_workspace.
template <typename T>
Nodes<T> mamba2_nodes(const WsLayout& w, void* workspace, bool has_lambda) {
  char* base = static_cast<char*>(workspace);
  Nodes<T> nodes{};
  nodes.t1 = reinterpret_cast<float*>(base + w.tot2);
  nodes.cl = reinterpret_cast<float*>(base + w.cl);
  if (has_lambda) {
    nodes.lvl1 = reinterpret_cast<T*>(base + w.lvl1);
    nodes.lvl2 = reinterpret_cast<T*>(base + w.lvl2);
    nodes.blocks = reinterpret_cast<T*>(base + w.blocks);
    nodes.upper = reinterpret_cast<T*>(base + w.upper);
    nodes.t2 = reinterpret_cast<float*>(base + w.t2);
    nodes.t3 = reinterpret_cast<float*>(base + w.t3);
    nodes.tup = reinterpret_cast<float*>(base + w.tup);
    nodes.n1 = w.n1;
    nodes.n2 = w.n2;
    nodes.nb = w.nb;
    nodes.nup = w.nup;
  }
  return nodes;
}

// Enqueues the forward's summary stages with lambda given (block_state, then the block-tree
// scan when the sequence has tile levels >= 4), filling `nodes`; `ev_mid`, when non-null, is
// recorded between the two.
template <typename T, int C, int DK, int DV>
hipError_t launch_mamba2_summaries(const Mamba2Args& a, const WsLayout& w, const Nodes<T>& nodes, hipStream_t st,
                                   hipEvent_t ev_mid);

// Kernel shapes (storage type, C, d_k, d_v) of the log-linear Mamba-2 kernels.
#define LL_MAMBA2_SHAPES(X)        \
  X(float, 16, 16, 16)             \
  X(float, 64, 64, 64)             \
  X(__bf16, 64, 64, 64)            \
  X(__bf16, 64, 128, 64)           \
  X(__bf16, 64, 128, 128)

}  // namespace ll
