// Log-linear Mamba-2 forward: O = (Q K^T (.) M^S (.) M^H) V  (Sec. 3.4), computed with the
// chunkwise algorithm of Sec. 3.3 (Eq. 5), organised for gfx950 in tiles of R = 2C tokens (at least 64).
//
// The hierarchical mask splits at the tile boundary exactly as Eq. 5 splits it at the chunk
// boundary: pairs (t, s) inside one aligned tile have levels 0..log2 R and are computed densely
// (the chunk-diagonal blocks D of Eq. 5 plus the two lowest inter-chunk levels, as one causal
// R x R masked contraction on MFMA); pairs in different tiles have level log2 R + j, where j is
// the bit length of (tile(t) XOR tile(s)), and are computed from summaries of whole source
// groups of tiles (the masked Q S products of the chunkwise algorithm, App. C Alg. 1).
//
// Kernels:
//   block_state  per block of 4 tiles: the tile states S_u = sum_t exp(tot_u - cl_t) v_t k_t^T
//                (MFMA, K = R tokens), folded on chip into the summaries the first three
//                tile levels read: S_u of even tiles (level 1), the pair summary of tiles 0-1
//                (level 2) and the whole-block summary (level 3), each with its summed log2-gate.
//   level_scan   per (b, h), elementwise over state entries: above the blocks the summaries form
//                a binary tree over the blocks of one sequence (tile level 3 + l for tree level
//                l), built chunk by chunk.  With lambda == NULL instead (running_scan): the
//                single running state entering every tile.
//   tile_out     per tile: the causal R x R masked contraction and, for every set bit j-1 of
//                the tile index, the lambda-weighted term  lambda_t^(log2 R + j) exp(cl_t + gap) q_t^T U_j,
//                gap_j being the summed totals of the tile's lower-level source groups.
//
// Decays are kept in the log2 domain (gates pre-multiplied by log2 e) and every exp2 argument
// is <= 0: tile-local cumulative sums and exact range sums of tile totals, never differences of
// sequence-long prefix sums.
#include <algorithm>
#include <type_traits>

#include "ll_fast_tile.hpp"
#include "ll_mamba2_common.hpp"

namespace ll {

// ---------------------------------------------------------------------------------------------
// Kernel 1: block states.  One workgroup (8 waves) per (block of 4 tiles, head, batch).  The
// gates of all the block's tiles are scanned once on entry (one row per thread); the K/V rows of
// the 64-row steps are loaded into registers two steps ahead of their use (two register buffers,
// across tile boundaries).  The steps are unrolled over the block, so that every step issues the
// same loads and stores and the waits for the loads can count them.  Finished summaries are
// staged in LDS and written with 16-byte stores.
// ---------------------------------------------------------------------------------------------
constexpr int kStateThreads = 512;  // block_state workgroup: 8 waves

template <typename T, int C, int DK, int DV, bool HAS_LAMBDA>
__global__ __launch_bounds__(kStateThreads) void k_block_state(const T* __restrict__ k, const T* __restrict__ v,
                                                     const float* __restrict__ log_alpha, Nodes<T> nodes,
                                                     T* __restrict__ tiles, float* __restrict__ tot2_out,
                                                     int64_t Tlen, int H, int Hqk) {
  using M = Mfma<T>;
  typedef typename Vec16<T>::type V16;
  constexpr int R = tile_rows(C);
  constexpr int LDV = DV + 16;   // row strides of the row-major V and (decay * K) tiles
  constexpr int LDK = DK + 16;
  constexpr int MT = DV / 16, NT = DK / 16;
  constexpr int NW = kStateThreads / 64;
  constexpr int WM = MT >= 2 ? 2 : 1;                            // waves along p
  constexpr int WN = (NW / WM) < NT ? (NW / WM) : NT;            // waves along n
  constexpr int TM = MT / WM, TN = NT / WN;                      // 16x16 tiles per wave
  constexpr int SZ = DK * DV;
  constexpr int VEC = Vec16<T>::N;
  constexpr int STEPS = R / kKB;                                 // 64-row steps per tile
  constexpr int GATES = kBlockTiles * R;                         // gate rows of a block
  static_assert(GATES <= kStateThreads && R % 64 == 0, "one gate row per thread, whole waves per tile");
  __shared__ T v_s[kKB * LDV];   // V rows of the current 64-row step
  __shared__ T k_s[kKB * LDK];   // decay * K rows
  __shared__ T out_s[2][SZ];     // summaries on their way out ([p][n], d_v x d_k)
  __shared__ float cl_s[GATES];  // per tile: inclusive cumulative log2-gates
  __shared__ float dec_s[GATES]; // per tile: decay from each row to the tile end (0 past it)
  __shared__ float wsum_s[NW];

  const int64_t N = (Tlen + R - 1) / R;  // tiles
  const int64_t NB = (N + kBlockTiles - 1) / kBlockTiles;
  const int64_t work = xcd_remap(blockIdx.x, (int64_t)gridDim.x);  // logical order (b, h, blk)
  const int blk = (int)(work % NB);
  const int64_t bh = work / NB;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int hq = h / (H / Hqk);  // this head's query/key head (heads share them in groups)
  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool active = wave < WM * WN;
  const int wm = wave / WN, wn = wave % WN;
  const int64_t u0 = (int64_t)blk * kBlockTiles;
  const int ntile = (int)((N - u0) < kBlockTiles ? (N - u0) : kBlockTiles);
  const int nsteps = ntile * STEPS;
  auto nrow_of = [&](int64_t u) { return (int)((Tlen - u * R) < R ? (Tlen - u * R) : R); };
  auto tile_row0 = [&](int64_t u) { return (int64_t)b * Tlen + u * R; };

  RowBlock<T, DK, kStateThreads> kr0, kr1;
  RowBlock<T, DV, kStateThreads> vr0, vr1;
  // loads of step s; past the last step the last one is loaded again (an L2 hit)
  auto load_step = [&](int s, RowBlock<T, DK, kStateThreads>& kr, RowBlock<T, DV, kStateThreads>& vr) {
    s = s < nsteps ? s : nsteps - 1;
    const int64_t u = u0 + s / STEPS;
    const int kb = s % STEPS;
    kr.load(k, tile_row0(u), kb * kKB, nrow_of(u), Hqk, hq);
    vr.load(v, tile_row0(u), kb * kKB, nrow_of(u), H, h);
  };

  // ---- gates of the block: thread tid holds row tid % R of tile tid / R
  {
    const int a = tid / R, r = tid % R;
    const int ac = a < ntile ? a : ntile - 1;
    const int nr = nrow_of(u0 + ac);
    const bool valid = tid < GATES && a < ntile && r < nr;
    const float la_raw = log_alpha[(tile_row0(u0 + ac) + (r < nr ? r : nr - 1)) * H + h];
    load_step(0, kr0, vr0);
    load_step(1, kr1, vr1);
    __builtin_amdgcn_sched_barrier(0);  // the gate's first use stays below the step loads
    float cl = wave_inclusive_scan(valid ? la_raw * kLog2e : 0.f);
    if (lane == 63) wsum_s[wave] = cl;
    __syncthreads();
    for (int w = (a * R) / 64; w < wave; ++w) cl += wsum_s[w];  // preceding waves of this tile
    if (tid < GATES) cl_s[tid] = cl;
    if (tid < GATES && a < ntile) nodes.cl[(bh * N + u0) * R + tid] = cl;
    __syncthreads();
    if (tid < GATES) dec_s[tid] = valid ? fast_exp2(cl_s[a * R + R - 1] - cl) : 0.f;
    if (tid < ntile) tot2_out[bh * N + u0 + tid] = cl_s[tid * R + R - 1];
  }

  f32x4 run[TM][TN], acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int jn = 0; jn < TN; ++jn) run[i][jn] = acc[i][jn] = f32x4{0.f, 0.f, 0.f, 0.f};

  // stage a summary (registers of the active waves) in out_s[slot]
  auto stage = [&](int slot, const f32x4 (&x)[TM][TN]) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int jn = 0; jn < TN; ++jn)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int p = (wm * TM + i) * 16 + 4 * g + r, n = (wn * TN + jn) * 16 + r16;
          out_s[slot][p * DK + n] = from_f32<T>(x[i][jn][r]);
        }
  };
  // (streaming stores: the summaries are read back by later kernels, not from the caches this
  // kernel's K/V stream passes through)
  auto flush = [&](int slot, T* dst) {
    constexpr int PASSES = (SZ / VEC + kStateThreads - 1) / kStateThreads;
#pragma unroll
    for (int it = 0; it < PASSES; ++it) {
      const int idx = tid + it * kStateThreads;
      if ((SZ / VEC) % kStateThreads == 0 || idx < SZ / VEC)
        __builtin_nontemporal_store(*reinterpret_cast<const V16*>(&out_s[slot][idx * VEC]),
                                    reinterpret_cast<V16*>(dst + idx * VEC));
    }
  };

  // step s = (tile a, 64-row step kb); a and kb are compile-time after unrolling
  auto step = [&](int a, int kb, RowBlock<T, DK, kStateThreads>& kr, RowBlock<T, DV, kStateThreads>& vr) {
    const int64_t u = u0 + a;
    if (kb == 0) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int jn = 0; jn < TN; ++jn) acc[i][jn] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    __syncthreads();  // previous step's readers done (and dec_s visible on entry)
    vr.store_rows(v_s, LDV);
    kr.store_rows_scaled(k_s, LDK, dec_s + a * R + kb * kKB);
    __syncthreads();
    load_step(a * STEPS + kb + 2, kr, vr);
    if (active) {
      // S^T[p][n] += sum_t V[t][p] (dK)[t][n]: both operands read down the token rows
#pragma unroll
      for (int ks = 0; ks < kKB / M::KSTEP; ++ks) {
        typename M::frag bf[TN];
#pragma unroll
        for (int jn = 0; jn < TN; ++jn) {
          const int n0 = (wn * TN + jn) * 16;
          if constexpr (M::KPL == 8) bf[jn] = frag_down_rows(k_s, LDK, ks * 32, n0);
          else bf[jn] = k_s[(ks * 4 + g) * LDK + n0 + r16];
        }
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int p0 = (wm * TM + i) * 16;
          typename M::frag af;
          if constexpr (M::KPL == 8) af = frag_down_rows(v_s, LDV, ks * 32, p0);
          else af = v_s[(ks * 4 + g) * LDV + p0 + r16];
#pragma unroll
          for (int jn = 0; jn < TN; ++jn) acc[i][jn] = M::mma(af, bf[jn], acc[i][jn]);
        }
      }
    }
    if (kb == STEPS - 1) {
      // tile done: fold it into the block's summaries and write the ones readers need
      T* dst0 = nullptr;
      T* dst1 = nullptr;
      if constexpr (HAS_LAMBDA) {
        const float e = fast_exp2(cl_s[a * R + R - 1]);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int jn = 0; jn < TN; ++jn) run[i][jn] = run[i][jn] * e + acc[i][jn];
        if ((a & 1) == 0) dst0 = nodes.at(bh, N, 1, u, SZ);                // even tile: its own state
        if (a == 1) dst1 = nodes.at(bh, N, 2, u - 1, SZ);                  // pair summary, tiles 0-1
        if (a == kBlockTiles - 1) dst1 = nodes.at(bh, N, 3, u - 3, SZ);    // block summary
        if (tid == 0 && a == 1) nodes.t2[bh * nodes.n2 + blk] = cl_s[R - 1] + cl_s[2 * R - 1];
        if (tid == 0 && a == kBlockTiles - 1) {
          float t = 0.f;
          for (int x = 0; x < kBlockTiles; ++x) t += cl_s[x * R + R - 1];
          nodes.t3[bh * nodes.nb + blk] = t;
        }
      } else {
        dst0 = tiles + (bh * N + u) * SZ;
      }
      if (active) {
        if (dst0) stage(0, acc);
        if (dst1) stage(1, run);
      }
      __syncthreads();
      if (dst0) flush(0, dst0);
      if (dst1) flush(1, dst1);
    }
  };

#pragma unroll
  for (int a = 0; a < kBlockTiles; ++a) {
    if (a >= ntile) break;
#pragma unroll
    for (int kb = 0; kb < STEPS; ++kb) {
      if (((a * STEPS + kb) & 1) == 0) step(a, kb, kr0, vr0);
      else step(a, kb, kr1, vr1);
    }
  }

}

// ---------------------------------------------------------------------------------------------
// Kernel 2 (lambda given): the block tree.  grid (d_v*d_k / 512, B * H); each thread owns two
// state entries of one (b, h).  Node (l, k) of tree level l >= 1 summarises blocks
// [k 2^l, (k + 1) 2^l):  node(l, k) = exp2(total of node(l-1, 2k+1)) node(l-1, 2k) + node(l-1, 2k+1).
// The blocks are taken in chunks of kScanChunk, a batch of chunks loaded together (128 block
// summaries for bf16: one load latency for a 512-tile sequence), the levels inside a chunk built
// in registers (fp32), and each level above accumulating the chunk nodes across chunks.
// Nodes some tile reads are stored (bf16 or the storage type).  The node totals come from a tree
// of block totals in LDS; workgroup x = 0 stores them.
// ---------------------------------------------------------------------------------------------
constexpr int kScanChunk = 32;      // blocks per chunk
constexpr int kScanChunkLevels = 5; // tree levels inside a chunk
constexpr int kScanThreads = 256;
constexpr int kScanBatch = 4;       // chunks whose loads are in flight together (bf16; half for fp32)

template <typename T, int LMAX>
__global__ __launch_bounds__(kScanThreads) void k_level_scan(Nodes<T> nodes, int64_t N, int J, int SZ) {
  typedef T T2 __attribute__((ext_vector_type(2)));
  constexpr int CB = kScanChunk, CL = kScanChunkLevels;
  extern __shared__ float tt_s[];  // totals tree: level 0 (blocks) first, then level 1, ...
  const int64_t bh = blockIdx.y;
  const int tid = threadIdx.x;
  const int64_t nb = nodes.nb;
  const int64_t nbp = (nb + CB - 1) / CB * CB;  // blocks rounded up to whole chunks
  const int LB = J - 3;                         // highest tree level with a read node
  const int LT = LB > CL ? LB : CL;             // levels of the totals tree (the chunk's at least)
  auto toff = [&](int l) {
    int64_t o = 0;
    for (int x = 0; x < l; ++x) o += (nbp + (int64_t(1) << x) - 1) >> x;
    return o;
  };
  // ---- totals tree (blocks past the last whole one count 0; no read node covers them)
  for (int64_t m = tid; m < nbp; m += kScanThreads) tt_s[m] = (m + 1) * kBlockTiles <= N ? nodes.t3[bh * nb + m] : 0.f;
  __syncthreads();
  for (int l = 1; l <= LT; ++l) {
    const int64_t o = toff(l), op = toff(l - 1), n = (nbp + (int64_t(1) << l) - 1) >> l;
    const int64_t np = (nbp + (int64_t(1) << (l - 1)) - 1) >> (l - 1);
    for (int64_t k = tid; k < n; k += kScanThreads)
      tt_s[o + k] = tt_s[op + 2 * k] + (2 * k + 1 < np ? tt_s[op + 2 * k + 1] : 0.f);
    __syncthreads();
  }
  auto tt = [&](int l, int64_t k) { return tt_s[toff(l) + k]; };
  if (blockIdx.x == 0) {
    for (int l = 1; l <= LB; ++l) {
      const int64_t n = (nbp + (int64_t(1) << l) - 1) >> l;
      for (int64_t k = tid; k < n; k += kScanThreads)
        if (tree_node_read(l, k, N)) nodes.tup[nodes.up_slot(bh, l, k)] = tt(l, k);
    }
  }
  const int e0 = (blockIdx.x * kScanThreads + tid) * 2;
  if (e0 >= SZ) return;

  const T* src = nodes.blocks + bh * nb * SZ + e0;
  auto store = [&](int l, int64_t k, float a0, float a1) {
    T2 out;
    out[0] = from_f32<T>(a0);
    out[1] = from_f32<T>(a1);
    *reinterpret_cast<T2*>(nodes.upper + nodes.up_slot(bh, l, k) * SZ + e0) = out;
  };
  auto load_chunk = [&](int64_t c, T2 (&x)[CB]) {
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int64_t m = c * CB + i < nb ? c * CB + i : nb - 1;
      x[i] = *reinterpret_cast<const T2*>(src + m * SZ);
    }
  };
  float acc0[LMAX + 1], acc1[LMAX + 1];  // levels above the chunk
#pragma unroll
  for (int l = 0; l <= LMAX; ++l) acc0[l] = acc1[l] = 0.f;
  auto use_chunk = [&](int64_t c, const T2 (&x)[CB]) {
    float v0[CB], v1[CB];
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      v0[i] = to_f32(x[i][0]);
      v1[i] = to_f32(x[i][1]);
    }
#pragma unroll
    for (int l = 1; l <= CL; ++l) {
#pragma unroll
      for (int i = 0; i < (CB >> l); ++i) {
        const int64_t k = ((c * CB) >> l) + i;
        const float e = fast_exp2(tt(l - 1, 2 * k + 1));
        v0[i] = e * v0[2 * i] + v0[2 * i + 1];
        v1[i] = e * v1[2 * i] + v1[2 * i + 1];
        if (l <= LB && tree_node_read(l, k, N)) store(l, k, v0[i], v1[i]);
      }
    }
    // v0[0], v1[0]: the whole chunk, node (CL, c)
#pragma unroll
    for (int l = CL + 1; l <= LMAX; ++l) {
      if (l > LB) break;
      const int sh = l - CL;
      const bool first = (c & ((int64_t(1) << sh) - 1)) == 0;
      const float e = first ? 0.f : fast_exp2(tt(CL, c));
      acc0[l] = acc0[l] * e + v0[0];
      acc1[l] = acc1[l] * e + v1[0];
      const int64_t k = c >> sh;
      if (((c + 1) & ((int64_t(1) << sh) - 1)) == 0 && tree_node_read(l, k, N)) store(l, k, acc0[l], acc1[l]);
    }
  };
  // batches of kScanBatch chunks: every load of a batch is issued before its first chunk is used
  constexpr int NBAT = kScanBatch * sizeof(__bf16) / sizeof(T);
  const int64_t nch = nbp / CB;
  for (int64_t c0 = 0; c0 < nch; c0 += NBAT) {
    T2 x[NBAT][CB];
#pragma unroll
    for (int bi = 0; bi < NBAT; ++bi)
      if (c0 + bi < nch) load_chunk(c0 + bi, x[bi]);
#pragma unroll
    for (int bi = 0; bi < NBAT; ++bi)
      if (c0 + bi < nch) use_chunk(c0 + bi, x[bi]);
  }
}

// ---------------------------------------------------------------------------------------------
// Kernel 2 (lambda == NULL only): running scan, elementwise over the d_v*d_k state entries
// (2 per thread), sequential over the tiles of one (b, h).
// ---------------------------------------------------------------------------------------------
constexpr int kScanUnroll = 8;      // summary loads in flight per thread

// lambda == NULL: the running state entering each tile, R_0 = 0, R_(u+1) = exp2(tot_u) R_u + S_u.
template <typename T>
__global__ __launch_bounds__(256) void k_running_scan(const T* __restrict__ tiles, T* __restrict__ running,
                                                      const float* __restrict__ tot2, int64_t N, int SZ) {
  typedef T T2 __attribute__((ext_vector_type(2)));
  extern __shared__ float dyn_s[];  // the N tile totals
  const int64_t bh = blockIdx.y;
  const int tid = threadIdx.x;
  for (int64_t u = tid; u < N; u += 256) dyn_s[u] = tot2[bh * N + u];
  __syncthreads();
  const int e0 = (blockIdx.x * 256 + tid) * 2;
  if (e0 >= SZ) return;
  const T* src = tiles + bh * N * SZ + e0;
  T* dst = running + bh * N * SZ + e0;
  float r0 = 0.f, r1 = 0.f;
  // batches of kScanUnroll tiles; the next batch's loads are issued before the current one is used
  auto load_batch = [&](int64_t u0, T2 (&sv)[kScanUnroll]) {
#pragma unroll
    for (int i = 0; i < kScanUnroll; ++i) {
      const int64_t u = u0 + i < N ? u0 + i : N - 1;
      sv[i] = *reinterpret_cast<const T2*>(src + u * SZ);
    }
  };
  auto use_batch = [&](int64_t u0, const T2 (&sv)[kScanUnroll]) {
#pragma unroll
    for (int i = 0; i < kScanUnroll; ++i) {
      if (u0 + i < N) {
        T2 out;
        out[0] = from_f32<T>(r0);
        out[1] = from_f32<T>(r1);
        *reinterpret_cast<T2*>(dst + (u0 + i) * SZ) = out;
        const float e = fast_exp2(dyn_s[u0 + i]);
        r0 = r0 * e + to_f32(sv[i][0]);
        r1 = r1 * e + to_f32(sv[i][1]);
      }
    }
  };
  T2 sa[kScanUnroll], sb[kScanUnroll];
  load_batch(0, sa);
  for (int64_t u0 = 0; u0 < N; u0 += 2 * kScanUnroll) {
    if (u0 + kScanUnroll < N) load_batch(u0 + kScanUnroll, sb);
    use_batch(u0, sa);
    if (u0 + kScanUnroll >= N) break;
    if (u0 + 2 * kScanUnroll < N) load_batch(u0 + 2 * kScanUnroll, sa);
    use_batch(u0 + kScanUnroll, sb);
  }
}

// ---------------------------------------------------------------------------------------------
// Kernel 3: tile outputs.  RS workgroups per (tile, head, batch), one wave per 16-row group.
//
// Work split: the R tile rows form R/16 groups of 16, one per wave.  With one workgroup per tile
// (R <= 128) wave w owns group w; with two (R = 256, 8 waves each) the groups pair up as
// (x, 15 - x), each pair costing 17 key tiles of the causal triangle, and the eight pairs are
// dealt to the two workgroups so that both do the same work.
// Orientation: the waves build O^T (d_v x rows) so that the query index is the MFMA column:
//   S^T = K Q^T per 16x16 tile (K = d_k), masked in registers with
//         lambda_i^(bitlen(i XOR j)) * exp2(cl_i - cl_j) for j <= i (tile-local i, j);
//   O^T += V^T P^T (P^T in the result layout of S^T is directly a B operand once V^T is
//         loaded at the same keys);
//   O^T += w (.) U^T Q^T for every inter-tile level (w = per-query weight, a column scale).
// The next 64-key block of K/V, and the next level's summary, are loaded into registers while
// the current one is being used.
// ---------------------------------------------------------------------------------------------
template <int R>
struct RowMap {
  static constexpr int RS = R >= 256 ? 2 : 1;   // workgroups per tile
  static constexpr int NW = R / 16 / RS;        // waves per workgroup: one 16-row group each
  static constexpr int NT = 64 * NW;            // threads per workgroup
  // 16-row group owned by `wave` of workgroup c
  __device__ static inline int group(int c, int wave) {
    if constexpr (RS == 1) {
      return wave;
    } else {
      // pairs (x, 15 - x); x in {0,3,4,7} -> workgroup 0, x in {1,2,5,6} -> workgroup 1;
      // waves 0-3 take x, waves 4-7 take 15 - x
      const int w4 = wave & 3;
      const int x = (c == 0) ? ((w4 & 1) ? 4 * (w4 >> 1) + 3 : 4 * (w4 >> 1))
                             : ((w4 & 1) ? 4 * (w4 >> 1) + 2 : 4 * (w4 >> 1) + 1);
      return wave < 4 ? x : (R / 16 - 1) - x;
    }
  }
};

// Matrix-valued level weights (the 4D-tensor view of App. A), LQ != 0: every 16 x 16 score tile
// is formed with the queries q_t Lambda_t^(l) of its own level -- one level for an off-diagonal
// key tile, levels 0-4 (selected per element) on the diagonal one, level log2 R + j for
// inter-tile level j -- and the scalar weights are 1.
//   LQ = 1: `q` holds those level queries, laid out [B, T, H, L, DK] (formed beforehand);
//   LQ = 2: diagonal Lambda: `q` is the plain query and `lam` the diagonals [B, T, H, L, DK]; the
//           level's query fragment is q (.) diag, rounded to T, formed in registers.
// Both read the Fenwick summaries (HAS_LAMBDA) and need H_qk = H.
// (the level-query forms hold a second query fragment set: two waves per SIMD, 256 registers)
template <typename T, int C, int DK, int DV, bool HAS_LAMBDA, int LQ = 0>
__global__ __launch_bounds__(RowMap<tile_rows(C)>::NT, LQ ? 2 : 4) void k_tile_out(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v, const float* __restrict__ log_alpha,
    const float* __restrict__ lam, Nodes<T> nodes, const T* __restrict__ running, T* __restrict__ o, int64_t Tlen,
    int H, int Hqk, int L, int J) {
  using M = Mfma<T>;
  typedef typename Vec16<T>::type V16;
  constexpr int R = tile_rows(C);
  constexpr int LOG2R = (R == 64) ? 6 : (R == 128) ? 7 : (R == 256) ? 8 : 9;
  constexpr int VEC = Vec16<T>::N;
  constexpr int LDK = DK + VEC;     // K and U row stride (elements)
  constexpr int LDV = DV + 16;      // V row stride (elements)
  using RM = RowMap<R>;
  constexpr int NT = RM::NT;
  constexpr int ROWS = 16 * RM::NW; // rows of this workgroup
  constexpr int MT = DV / 16, KS = DK / M::KSTEP;
  constexpr int SZ = DK * DV;
  constexpr int KV_ELEMS = kKB * LDK + kKB * LDV;
  constexpr int U_ELEMS = DV * LDK;
  constexpr int ULOADS = (SZ / VEC + NT - 1) / NT;
  __shared__ T buf_s[KV_ELEMS > U_ELEMS ? KV_ELEMS : U_ELEMS];
  __shared__ float cl_s[R];
  __shared__ float wsum_s[4];
  static_assert(LQ == 0 || HAS_LAMBDA, "level queries read the Fenwick summaries");
  constexpr bool STAGE_LAMBDA = HAS_LAMBDA && LQ == 0;
  __shared__ float lam_s[STAGE_LAMBDA ? ROWS * kMaxLevels : 1];  // row 16 * wave + r16 of this workgroup
  __shared__ float kdec_s[R];
  T* k_s = buf_s;
  T* v_s = buf_s + kKB * LDK;
  T* u_s = buf_s;

  const int64_t N = (Tlen + R - 1) / R;
  const int64_t work = xcd_remap(blockIdx.x, (int64_t)gridDim.x);  // logical order (b, h, u, c)
  const int c = (int)(work % RM::RS);
  const int u = (int)((work / RM::RS) % N);
  const int64_t bh = work / (RM::RS * N);
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int hq = h / (H / Hqk);  // this head's query/key head
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, r16 = lane & 15, g = lane >> 4;
  const int64_t row0 = (int64_t)b * Tlen + (int64_t)u * R;
  const int nrow = (int)((Tlen - (int64_t)u * R) < R ? (Tlen - (int64_t)u * R) : R);
  const int nkb = (nrow + kKB - 1) / kKB;
  const int gi = RM::group(c, wave);             // this wave's 16-row group
  const int i = 16 * gi + r16;                   // this lane's row (tile-local)
  const int nkb_w = (16 * gi + 15) / kKB + 1;    // key blocks this wave's rows reach

  RowBlock<T, DK, NT> kr;
  RowBlock<T, DV, NT> vr;
  kr.load(k, row0, 0, nrow, Hqk, hq);
  vr.load(v, row0, 0, nrow, H, h);
  const float la = tile_gate<R>(log_alpha, row0, nrow, H, h);  // issued with the other loads

  // Q^T fragments (B operand) of this lane's row, kept in registers (LQ: of one level at a time,
  // qlev naming it; LQ = 2 keeps the plain query in qbase).  With LQ, a level's data is fetched
  // (fetch_q: LQ = 1 the level-query fragments, LQ = 2 the diagonal's entries of this lane's k
  // slots, zeros for rows past the end) and then turned into qf (form_q), so that the inter-tile
  // loop can fetch the next level while the current one runs.
  typename M::frag qf[KS], qbase[LQ == 2 ? KS : 1], qraw[LQ == 1 ? KS : 1];
  float wraw[LQ == 2 ? KS * M::KPL : 1];
  int qlev = 0;
  auto fetch_q = [&](int l) {
    if constexpr (LQ == 2) {
      const float* wsrc = lam + (((row0 + i) * H + h) * L + l) * DK + g * M::KPL;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if constexpr (M::KPL == 8) {
          const f32x4 z4 = {0.f, 0.f, 0.f, 0.f};
          const f32x4 w0 = i < nrow ? *reinterpret_cast<const f32x4*>(wsrc + ks * M::KSTEP) : z4;
          const f32x4 w1 = i < nrow ? *reinterpret_cast<const f32x4*>(wsrc + ks * M::KSTEP + 4) : z4;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            wraw[ks * 8 + e] = w0[e];
            wraw[ks * 8 + 4 + e] = w1[e];
          }
        } else {
          wraw[ks] = i < nrow ? wsrc[ks * M::KSTEP] : 0.f;
        }
      }
    } else if constexpr (LQ == 1) {
      const T* src = q + (((row0 + i) * H + h) * L + l) * DK;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qraw[ks] = i < nrow ? M::load(src + ks * M::KSTEP + g * M::KPL) : typename M::frag{};
    }
  };
  auto form_q = [&](int l) {
    if constexpr (LQ == 2) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if constexpr (M::KPL == 8) {
#pragma unroll
          for (int e = 0; e < 8; ++e) qf[ks][e] = from_f32<T>(to_f32(qbase[ks][e]) * wraw[ks * 8 + e]);
        } else {
          qf[ks] = from_f32<T>(to_f32(qbase[ks]) * wraw[ks]);
        }
      }
    } else if constexpr (LQ == 1) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) qf[ks] = qraw[ks];
    }
    qlev = l;
  };
  auto load_q = [&](int l) {
    if constexpr (LQ != 0) {
      fetch_q(l);
      form_q(l);
    } else {
      const T* src = q + ((row0 + i) * Hqk + hq) * DK;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qf[ks] = i < nrow ? M::load(src + ks * M::KSTEP + g * M::KPL) : typename M::frag{};
      qlev = l;
    }
  };
  if constexpr (LQ == 2) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qbase[ks] = i < nrow ? M::load(q + ((row0 + i) * H + h) * DK + ks * M::KSTEP + g * M::KPL) : typename M::frag{};
  }
  // LQ: the level of this wave's first key tile is fetched now, formed when the tile comes
  int pre = -1;
  if constexpr (LQ != 0) {
    qlev = -1;
    pre = gi > 0 ? level_local(16 * gi, 0) : 0;
    fetch_q(pre);
  } else {
    load_q(0);
  }
  if constexpr (STAGE_LAMBDA) {
    // one row of lambda per thread of the first ROWS threads, loads issued before the stores
    if (tid < ROWS) {
      const int row = 16 * RM::group(c, tid >> 4) + (tid & 15);
      if (row < nrow) {
        const float* src = lam + ((row0 + row) * H + h) * L;
#pragma unroll
        for (int l0 = 0; l0 < kMaxLevels; l0 += kMaxLevels / 3) {  // three batches of loads
          float lv[kMaxLevels / 3];
#pragma unroll
          for (int l = 0; l < kMaxLevels / 3; ++l)
            if (l0 + l < L) lv[l] = src[l0 + l];
#pragma unroll
          for (int l = 0; l < kMaxLevels / 3; ++l)
            if (l0 + l < L) lam_s[tid * L + l0 + l] = lv[l];
        }
      }
    }
  }
  tile_cumsum_of<R>(la, nrow, cl_s, wsum_s);
  // key-side decay to the end of each 16-key tile: kdec[j] = exp2(cl[j | 15] - cl[j])
  for (int r = tid; r < R; r += NT) kdec_s[r] = fast_exp2(cl_s[r | 15] - cl_s[r]);
  const float* lrow = STAGE_LAMBDA ? &lam_s[(16 * wave + r16) * L] : lam_s;  // this lane's lambda row

  // ---- summaries of the inter-tile levels (set bits of u); the first one is prefetched while
  //      the last key block is being used, each next one while the current level is
  float gapv = 0.f;
  if constexpr (HAS_LAMBDA) gapv = level_gaps(nodes, bh, N, u, J);
  auto level_src = [&](int j, float* gap) -> const T* {
    if constexpr (HAS_LAMBDA) {
      *gap = gap_of(gapv, j);
      return nodes.at(bh, N, j, source_first(u, j), SZ);
    } else {
      *gap = 0.f;
      return running + (bh * N + u) * SZ;
    }
  };
  auto next_level = [&](int j) {
    if constexpr (HAS_LAMBDA) {
      for (++j; j <= J; ++j)
        if (reads_level(u, j)) return j;
      return 0;
    } else {
      return (j == 0 && u > 0) ? 1 : 0;
    }
  };
  V16 ur[ULOADS];
  auto load_u = [&](const T* U) {
#pragma unroll
    for (int e = 0; e < ULOADS; ++e) {
      const int idx = tid + NT * e;
      if (idx < SZ / VEC) ur[e] = *reinterpret_cast<const V16*>(U + idx * VEC);
    }
  };
  int j = next_level(0);
  float gap = 0.f;

  f32x4 oacc[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) oacc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // ---- intra-tile: causal R x R masked contraction, one 64-key block at a time
  for (int kb = 0; kb < nkb; ++kb) {
    __syncthreads();  // previous block's readers are done (and cl/lambda staging on entry)
    kr.store_rows(k_s, LDK);
    vr.store_rows(v_s, LDV);
    __syncthreads();
    if (kb + 1 < nkb) {
      kr.load(k, row0, (kb + 1) * kKB, nrow, Hqk, hq);
      vr.load(v, row0, (kb + 1) * kKB, nrow, H, h);
    } else if (HAS_LAMBDA && j) {
      load_u(level_src(j, &gap));
    }
    if (kb >= nkb_w || 16 * gi >= nrow) continue;
    const float cli = cl_s[i];
    // key sub-steps: 32 keys (bf16, two 16-key tiles) or 16 keys (fp32)
    constexpr int KT_PER = (M::KPL == 8) ? 2 : 1;
#pragma unroll
    for (int st = 0; st < 4 / KT_PER; ++st) {
      const int KT0 = 4 * kb + st * KT_PER;  // first 16-key tile of the sub-step (tile-local)
      if (KT0 > gi) break;
      f32x4 p[KT_PER];
#pragma unroll
      for (int hh = 0; hh < KT_PER; ++hh) {
        const int kt = st * KT_PER + hh, KT = KT0 + hh;
        p[hh] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (KT > gi) continue;
        f32x4 sacc = {0.f, 0.f, 0.f, 0.f};
        auto scores = [&]() {
          f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            acc = M::mma(M::load(&k_s[(kt * 16 + r16) * LDK + ks * M::KSTEP + g * M::KPL]), qf[ks], acc);
          return acc;
        };
        if constexpr (LQ != 0) {
          if (KT < gi) {
            const int lv = level_local(16 * gi, 16 * KT);
            if (lv != qlev) {
              if (pre == lv) form_q(lv);
              else load_q(lv);
              // fetch the next level this wave's key tiles reach: as KT grows the highest bit in
              // which KT differs from gi (level 5 + that bit) steps down the set bits of gi, and
              // after the last one comes the diagonal tile (level 0)
              const int below = gi & ((1 << (lv - 5)) - 1);
              pre = below ? 4 + bitlen(uint32_t(below)) : 0;
              fetch_q(pre);
            }
            sacc = scores();
          } else {
            // diagonal 16 x 16 tile: pairs at levels 0-4, each scored with its level's queries,
            // the next level fetched while the current one is scored
            if (pre != 0) fetch_q(0);
            f32x4 sl[5];
#pragma unroll
            for (int l = 0; l < 5; ++l) {
              form_q(l);
              if (l + 1 < 5) fetch_q(l + 1);
              sl[l] = scores();
            }
            pre = -1;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int j = 16 * KT + 4 * g + r, lv = level_local(i, j);
              float x = 0.f;
#pragma unroll
              for (int l = 0; l < 5; ++l) x = lv == l ? sl[l][r] : x;
              p[hh][r] = j <= i ? x * fast_exp2(cli - cl_s[j]) : 0.f;
            }
            continue;
          }
        } else {
          sacc = scores();
        }
        if (KT < gi) {
          // off-diagonal 16x16 tile: one level for the whole tile (4 + bitlen(gi ^ KT)) and the
          // decay split at the tile's last key: exp2(cl_i - cl_end) * exp2(cl_end - cl_j)
          float qs = fast_exp2(cli - cl_s[16 * KT + 15]);
          if constexpr (STAGE_LAMBDA) qs *= lrow[level_local(16 * gi, 16 * KT)];
          const f32x4 kd = *reinterpret_cast<const f32x4*>(&kdec_s[16 * KT + 4 * g]);
#pragma unroll
          for (int r = 0; r < 4; ++r) p[hh][r] = sacc[r] * qs * kd[r];
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int j = 16 * KT + 4 * g + r;
            float w = 0.f;
            if (j <= i) {
              w = fast_exp2(cli - cl_s[j]);
              if constexpr (STAGE_LAMBDA) w *= lrow[level_local(i, j)];
            }
            p[hh][r] = sacc[r] * w;
          }
        }
      }
      if constexpr (M::KPL == 8) {
        // slots 0-3 <- key tile KT0 rows 4g..4g+3, slots 4-7 <- key tile KT0+1 rows 4g..4g+3;
        // the V^T fragment is read down the same key rows of the row-major V tile.
        typename M::frag bp;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          bp[r] = from_f32<T>(p[0][r]);
          bp[4 + r] = from_f32<T>(p[1][r]);
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) oacc[mt] = M::mma(frag_down_rows(v_s, LDV, st * 32, mt * 16), bp, oacc[mt]);
      } else {
        // fp32: one k step = 4 keys {16 kt + 4g + r : g}, i.e. slot r of every lane group.
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
            oacc[mt] = M::mma(v_s[(st * 16 + 4 * g + r) * LDV + mt * 16 + r16], p[0][r], oacc[mt]);
      }
    }
  }

  if (!HAS_LAMBDA && j) load_u(level_src(j, &gap));
  if constexpr (LQ != 0) {
    if (j) fetch_q(LOG2R + j);
  }
  while (j) {
    __syncthreads();  // LDS buffer free
#pragma unroll
    for (int e = 0; e < ULOADS; ++e) {
      const int idx = tid + NT * e;
      if (idx < SZ / VEC) {
        const int p = idx / (DK / VEC), n0 = (idx % (DK / VEC)) * VEC;
        *reinterpret_cast<V16*>(&u_s[p * LDK + n0]) = ur[e];
      }
    }
    __syncthreads();
    const int jn = next_level(j);
    float gap_n = 0.f;
    if (jn) load_u(level_src(jn, &gap_n));
    float w = fast_exp2(cl_s[i] + gap);
    if constexpr (STAGE_LAMBDA) w *= (i < nrow) ? lrow[LOG2R + j] : 0.f;
    if constexpr (LQ != 0) {
      form_q(LOG2R + j);                   // fetched one level ahead
      if (jn) fetch_q(LOG2R + jn);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      f32x4 tmp = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        tmp = M::mma(M::load(&u_s[(mt * 16 + r16) * LDK + ks * M::KSTEP + g * M::KPL]), qf[ks], tmp);
      oacc[mt] += w * tmp;
    }
    j = jn;
    gap = gap_n;
  }

  // ---- store O: lane holds row i, d_v entries 16 mt + 4g .. +3
  if (i < nrow) {
    T* orow = o + ((row0 + i) * H + h) * DV + 4 * g;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) orow[mt * 16 + r] = from_f32<T>(oacc[mt][r]);
  }
}

// ---------------------------------------------------------------------------------------------
// Kernel 3, bf16 tiles of R = 128 rows (C = 64): tile outputs with the tile's K and V resident
// in LDS.  One workgroup of 4 waves per (tile, head, batch).
//
// Wave w owns the 16-row groups w and 7 - w (32 rows): each wave covers 9 of the 36 key tiles of
// the causal triangle and 32 rows of every inter-tile level, and every K, V or summary fragment
// it reads from LDS feeds two MFMAs (one per group).  Orientation as in k_tile_out (O^T built
// with the query index as the MFMA column).
//
// K, V and the level summaries are copied straight from global memory into LDS
// (global_load_lds_dwordx4: lane l of a wave instruction writes bytes 16 l .. 16 l + 15 of a 1 KiB
// span), into row-major tiles whose 16-byte chunks are XOR-swizzled by row: chunk c of row r sits
// at position c ^ (r mod chunks-per-row), so a fragment read down 16 consecutive rows touches 16
// different chunk positions.  With the whole tile resident, the intra-tile phase runs without a
// barrier; the inter-tile levels alternate between the K and V regions, the next level's summary
// being copied in while the current one is used.
// ---------------------------------------------------------------------------------------------
template <int DK, int DV, bool HAS_LAMBDA>
__global__ __launch_bounds__(kFastThreads, 2) void k_tile_out_fast(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    const float* __restrict__ log_alpha, const float* __restrict__ lam, Nodes<__bf16> nodes,
    const __bf16* __restrict__ running, __bf16* __restrict__ o, int64_t Tlen,
    int H, int Hqk, int L, int J) {
  using M = Mfma<__bf16>;
  typedef __bf16 bf;
  typedef typename M::frag frag;
  constexpr int R = kFastRows, LOG2R = 7;
  constexpr int NT = kFastThreads;
  constexpr int MT = DV / 16, KS = DK / M::KSTEP, KC = M::KSTEP / 8;  // KC: 16-byte chunks per k step
  constexpr int SZ = DK * DV;
  static_assert(DK <= R && DV <= R, "a summary must fit in the K and in the V region");
  __shared__ bf k_s[R * DK];
  __shared__ bf v_s[R * DV];
  __shared__ float lam_s[HAS_LAMBDA ? R * kMaxLevels : 1];
  __shared__ float cl_s[R];
  __shared__ float kdec_s[R];

  const int64_t N = (Tlen + R - 1) / R;
  const int64_t work = xcd_remap(blockIdx.x, (int64_t)gridDim.x);  // logical order (b, h, u)
  const int u = (int)(work % N);
  const int64_t bh = work / N;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int hq = h / (H / Hqk);  // this head's query/key head
  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t row0 = (int64_t)b * Tlen + (int64_t)u * R;
  const int nrow = (int)((Tlen - (int64_t)u * R) < R ? (Tlen - (int64_t)u * R) : R);
  const int gA = wave, gB = 7 - wave;          // this wave's 16-row groups
  const int iA = 16 * gA + r16, iB = 16 * gB + r16;
  const bool liveB = 16 * gB < nrow;           // nrow is a multiple of C = 64

  // ---- loads: the tile's cumulative log2-gates (written by block_state) first, then Q into
  //      registers, then K, V, lambda into LDS
  lds_gather4<NT>(cl_s, R, [&](int x) { return nodes.cl + (bh * N + u) * R + x; });
  frag qA[KS], qB[KS];
  {
    const int rA = iA < nrow ? iA : nrow - 1, rB = iB < nrow ? iB : nrow - 1;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      qA[ks] = M::load(q + ((row0 + rA) * Hqk + hq) * DK + ks * M::KSTEP + g * M::KPL);
      qB[ks] = M::load(q + ((row0 + rB) * Hqk + hq) * DK + ks * M::KSTEP + g * M::KPL);
    }
  }
  lds_copy_rows<DK, R, NT>(k_s, k + (row0 * Hqk + hq) * DK, (int64_t)Hqk * DK, nrow);
  lds_copy_rows<DV, R, NT>(v_s, v + (row0 * H + h) * DV, (int64_t)H * DV, nrow);
  if constexpr (HAS_LAMBDA) lds_copy_lambda<R, NT>(lam_s, lam, row0, H, h, L, nrow);
  // decay gaps of the tile's levels, lane j - 1 holding level j's
  float gapv = 0.f;
  if constexpr (HAS_LAMBDA) gapv = level_gaps(nodes, bh, N, u, J);
  wait_vmem();
  __syncthreads();  // gates, K, V, lambda visible
  for (int r = tid; r < R; r += NT) kdec_s[r] = fast_exp2(cl_s[r | 15] - cl_s[r]);
  __syncthreads();  // kdec visible
  if (!liveB) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qB[ks] = frag{};  // rows past the end contribute nothing
  }

  // ---- intra-tile: causal 128 x 128 masked contraction, 32 keys per step, no barrier.  The
  //      body is instantiated per wave (groups GA = wave, GB = 7 - wave known at compile time),
  //      so that every skipped key tile and every mask case is resolved statically.
  const float cliA = cl_s[iA], cliB = cl_s[iB];
  const float* lrowA = &lam_s[HAS_LAMBDA ? iA * kMaxLevels : 0];
  const float* lrowB = &lam_s[HAS_LAMBDA ? iB * kMaxLevels : 0];
  f32x4 oA[MT], oB[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) oA[mt] = oB[mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  fast_intra<DK, DV, HAS_LAMBDA>(wave, k_s, v_s, cl_s, kdec_s, qA, qB, cliA, cliB, lrowA, lrowB, oA, oB);

  // ---- inter-tile levels (set bits of u): summaries alternate between the K and V regions
  auto level_src = [&](int j, float* gap) -> const bf* {
    if constexpr (HAS_LAMBDA) {
      *gap = gap_of(gapv, j);
      return nodes.at(bh, N, j, source_first(u, j), SZ);
    } else {
      *gap = 0.f;
      return running + (bh * N + u) * SZ;
    }
  };
  auto next_level = [&](int j) {
    if constexpr (HAS_LAMBDA) {
      for (++j; j <= J; ++j)
        if (reads_level(u, j)) return j;
      return 0;
    } else {
      return (j == 0 && u > 0) ? 1 : 0;
    }
  };
  // One level from `cur` (already being copied in); the next level's summary goes to `nxt`.
  auto level_step = [&](int& j, float& gap, const bf* cur, bf* nxt) {
    wait_vmem();
    __syncthreads();  // `cur` complete and visible; every wave is done with `nxt`
    const int jn = next_level(j);
    float gap_n = 0.f;
    if (jn) lds_copy_rows<DK, DV, NT>(nxt, level_src(jn, &gap_n), DK, DV);
    float wA = fast_exp2(cliA + gap), wB = fast_exp2(cliB + gap);
    if constexpr (HAS_LAMBDA) {
      wA *= lrowA[LOG2R + j];
      wB *= lrowB[LOG2R + j];
    }
    // summary fragments read one 16-row block ahead of their use
    frag uf[2][KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) uf[0][ks] = frag_along_row_swz<DK>(cur, 0, ks * KC);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      if (mt + 1 < MT) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) uf[(mt + 1) & 1][ks] = frag_along_row_swz<DK>(cur, 16 * (mt + 1), ks * KC);
      }
      f32x4 tA = {0.f, 0.f, 0.f, 0.f}, tB = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        tA = M::mma(uf[mt & 1][ks], qA[ks], tA);
        tB = M::mma(uf[mt & 1][ks], qB[ks], tB);
      }
      oA[mt] += wA * tA;
      oB[mt] += wB * tB;
    }
    j = jn;
    gap = gap_n;
  };

  int j = next_level(0);
  float gap = 0.f;
  __syncthreads();  // every wave is done with K and V
  if (j) lds_copy_rows<DK, DV, NT>(k_s, level_src(j, &gap), DK, DV);
  while (j) {
    level_step(j, gap, k_s, v_s);
    if (!j) break;
    level_step(j, gap, v_s, k_s);
  }

  // ---- store O through LDS: the lane's pieces (rows iA, iB, d_v entries 16 mt + 4g .. +3) go to
  //      a swizzled row-major tile in the V region, then whole rows leave as 16-byte pieces, 16
  //      consecutive lanes per 256-byte row
  __syncthreads();  // every wave is done with the last summary
  auto stage_rows = [&](const f32x4* acc, int i) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      bf16x4 val;
#pragma unroll
      for (int r = 0; r < 4; ++r) val[r] = from_f32<bf>(acc[mt][r]);
      *reinterpret_cast<bf16x4*>(v_s + swz<DV>(i, 2 * mt + (g >> 1)) + 4 * (g & 1)) = val;
    }
  };
  stage_rows(oA, iA);
  stage_rows(oB, iB);
  __syncthreads();
  constexpr int OCH = DV / 8;  // 16-byte pieces per row
#pragma unroll
  for (int it = 0; it < R * OCH / NT; ++it) {
    const int idx = it * NT + tid, r = idx / OCH, c = idx % OCH;
    if (r < nrow)
      *reinterpret_cast<bf16x8*>(o + ((row0 + r) * H + h) * DV + 8 * c) = *reinterpret_cast<const bf16x8*>(v_s + swz<DV>(r, c));
  }
}

// ---------------------------------------------------------------------------------------------
// Debug level map: the level each (t, s) pair receives from the device functions the kernels use.
// ---------------------------------------------------------------------------------------------
// Inside a tile the level is evaluated both as the generic tile kernels pick it (level_local) and, for
// tiles of 128 rows, as the 16 x 16 MFMA tiles of the fast and single-pass kernels pick it; across
// tiles both by the source-group start (three-kernel forward, backward) and by the group end (the
// single-pass forward walks the set bits of the tile index from the highest).  A pair the two
// decompositions disagree on is written as -3, a pair no group claims as -2.
__global__ void k_debug_level_map(int64_t Tlen, int R, int log2R, int J, int8_t* out) {
  const int64_t t = blockIdx.x;
  for (int64_t s = threadIdx.x; s < Tlen; s += blockDim.x) {
    int lev = -1;
    if (s <= t) {
      const int64_t ut = t / R, us = s / R;
      if (ut == us) {
        const int i = int(t % R), j = int(s % R);
        lev = level_local(i, j);
        if (R == 128) {
          const int fast = (i >> 4) == (j >> 4) ? level_in_group(i & 15, j & 15) : level_across_groups(i >> 4, j >> 4);
          if (fast != lev) lev = -3;
        }
      } else {
        lev = -2;  // no source group claims the pair: a bug
        for (int j = 1; j <= J; ++j)
          if (reads_level(ut, j) && us >= source_first(ut, j) && us < source_first(ut, j) + (int64_t(1) << (j - 1)))
            lev = log2R + j;
        int byend = -2;
        for (int j = ut ? bitlen(uint32_t(ut)) : 0; j >= 1; --j)
          if (((ut >> (j - 1)) & 1) && us < group_end(ut, j) && us >= group_end(ut, j) - (int64_t(1) << (j - 1)))
            byend = log2R + j;
        if (byend != lev) lev = -3;
      }
    }
    out[t * Tlen + s] = (int8_t)lev;
  }
}

// ---------------------------------------------------------------------------------------------
// Level queries for full matrix-valued level weights (App. A): qlev[row, l, :] = q[row, :] Lambda
// with Lambda = lam[row, l] (laid out [rows, L, DK, DK], (q Lambda)_c = sum_a q_a lam[row, l, a, c])
// for every row (b, t, h) and level l < L, rounded once to the storage type.  One wave per
// (row, level): lane c accumulates columns c and c + 64, each step a reading one coalesced row of
// Lambda, with q_a broadcast from the lane that loaded it.  (Diagonal weights need no such pass:
// the tile kernel scales its query fragments in registers.)
// ---------------------------------------------------------------------------------------------
constexpr int kLevelQueryThreads = 256;

template <typename T, int DK>
__global__ __launch_bounds__(kLevelQueryThreads) void k_level_queries_full(const T* __restrict__ q,
                                                                           const float* __restrict__ lam,
                                                                           T* __restrict__ qlev, int64_t rows, int L) {
  constexpr int CPL = (DK + 63) / 64;  // columns (and q entries) per lane
  const int lane = threadIdx.x & 63;
  const int64_t rl = blockIdx.x * (int64_t)(kLevelQueryThreads / 64) + (threadIdx.x >> 6);
  if (rl >= rows * L) return;  // whole waves leave together
  const int64_t row = rl / L;
  float qa[CPL], acc[CPL];
#pragma unroll
  for (int e = 0; e < CPL; ++e) {
    const int a = lane + 64 * e;
    qa[e] = a < DK ? to_f32(q[row * DK + a]) : 0.f;
    acc[e] = 0.f;
  }
  const float* m = lam + rl * DK * DK;
  constexpr int AN = DK < 64 ? DK : 64;  // q entries held per lane slot
#pragma unroll
  for (int ea = 0; ea < CPL; ++ea) {
#pragma unroll 4
    for (int a0 = 0; a0 < AN; ++a0) {
      const int a = 64 * ea + a0;
      const float qv = __shfl(qa[ea], a0, 64);
#pragma unroll
      for (int e = 0; e < CPL; ++e) {
        const int c = lane + 64 * e;
        if (c < DK) acc[e] += qv * m[a * DK + c];
      }
    }
  }
#pragma unroll
  for (int e = 0; e < CPL; ++e) {
    const int c = lane + 64 * e;
    if (c < DK) qlev[rl * DK + c] = from_f32<T>(acc[e]);
  }
}

// ---------------------------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------------------------
static int bitlen_h(uint64_t x) { return x ? 64 - __builtin_clzll(x) : 0; }

int64_t tiles_of(int64_t T, int64_t C) { return (T + tile_rows((int)C) - 1) / tile_rows((int)C); }

int tile_levels(int64_t T, int64_t C) {
  const int64_t N = tiles_of(T, C);
  return N <= 1 ? 0 : bitlen_h(uint64_t(N - 1));
}

int64_t mamba2_workspace(int64_t B, int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t C, int64_t esize,
                         bool has_lambda, WsLayout* lay) {
  const int64_t N = tiles_of(T, C);
  const int J = tile_levels(T, C);
  const int64_t BH = B * H, SZ = dk * dv;
  auto al = [](int64_t x) { return (x + 255) & ~int64_t(255); };
  WsLayout w{};
  w.N = N;
  w.J = J;
  w.n1 = (N + 1) / 2;
  w.n2 = (N + 3) / 4;
  w.nb = (N + kBlockTiles - 1) / kBlockTiles;
  w.nup = 0;
  for (int l = 1; l <= J - 3; ++l) w.nup += (w.nb + (int64_t(1) << l) - 1) >> l;  // block-tree levels
  const int64_t nup1 = w.nup > 0 ? w.nup : 1;
  int64_t cur = 0;
  w.tag = cur; cur += al(sizeof(WsTag));
  w.tot2 = cur; cur += al(BH * N * 4);
  w.cl = cur; cur += al(BH * N * tile_rows((int)C) * 4);
  if (has_lambda) {
    w.t2 = cur; cur += al(BH * w.n2 * 4);
    w.t3 = cur; cur += al(BH * w.nb * 4);
    w.tup = cur; cur += al(BH * nup1 * 4);
    w.lvl1 = cur; cur += al(BH * w.n1 * SZ * esize);
    w.lvl2 = cur; cur += al(BH * w.n2 * SZ * esize);
    w.blocks = cur; cur += al(BH * w.nb * SZ * esize);
    w.upper = cur; cur += al(BH * nup1 * SZ * esize);
  } else {
    w.tiles = cur; cur += al(BH * N * SZ * esize);
    w.running = cur; cur += al(BH * N * SZ * esize);
  }
  w.total = cur;
  if (lay) *lay = w;
  return cur;
}

__global__ void k_write_tag(uint64_t* dst, WsTag tag) {
  if (threadIdx.x < 12) dst[threadIdx.x] = tag.v[threadIdx.x];
}

WsTag mamba2_tag(const Mamba2Args& a, int64_t esize, bool valid) {
  WsTag t{};
  t.v[0] = valid ? kWsTagMagic : 0;
  t.v[1] = (uint64_t)a.B;
  t.v[2] = (uint64_t)a.T;
  t.v[3] = (uint64_t)a.H;
  t.v[4] = (uint64_t)a.Hqk;
  t.v[5] = (uint64_t)a.dk;
  t.v[6] = (uint64_t)a.dv;
  t.v[7] = (uint64_t)a.C;
  t.v[8] = (uint64_t)esize;
  t.v[9] = (uint64_t)(uintptr_t)a.k;
  t.v[10] = (uint64_t)(uintptr_t)a.v;
  t.v[11] = (uint64_t)(uintptr_t)a.log_alpha;
  return t;
}

hipError_t launch_write_tag_at(void* dst, const WsTag& tag, hipStream_t st) {
  hipLaunchKernelGGL(k_write_tag, dim3(1), dim3(64), 0, st, static_cast<uint64_t*>(dst), tag);
  return hipGetLastError();
}

hipError_t launch_write_tag(void* workspace, const WsLayout& w, const WsTag& tag, hipStream_t st) {
  return launch_write_tag_at(static_cast<char*>(workspace) + w.tag, tag, st);
}

// Also records, once the summaries are complete, the tag of the inputs they were formed from.
template <typename T, int C, int DK, int DV>
hipError_t launch_mamba2_summaries(const Mamba2Args& a, const WsLayout& w, const Nodes<T>& nodes, hipStream_t st,
                                   hipEvent_t ev_mid) {
  constexpr int SZ = DK * DV;
  const dim3 gblk((unsigned)(w.nb * a.H * a.B));
  hipLaunchKernelGGL((k_block_state<T, C, DK, DV, true>), gblk, dim3(kStateThreads), 0, st, (const T*)a.k, (const T*)a.v,
                     a.log_alpha, nodes, (T*)nullptr, const_cast<float*>(nodes.t1), a.T, (int)a.H, (int)a.Hqk);
  if (ev_mid) (void)hipEventRecord(ev_mid, st);
  if (w.J >= 4) {
    // LDS: the totals tree (the block count rounded up to whole chunks, and its levels)
    const int64_t nbp = (w.nb + kScanChunk - 1) / kScanChunk * kScanChunk;
    int64_t tt = 0;
    const int lt = w.J - 3 > kScanChunkLevels ? w.J - 3 : kScanChunkLevels;
    for (int l = 0; l <= lt; ++l) tt += (nbp + (int64_t(1) << l) - 1) >> l;
    const dim3 glev((unsigned)((SZ + 2 * kScanThreads - 1) / (2 * kScanThreads)), (unsigned)(a.B * a.H));
    if (w.J - 3 <= kScanChunkLevels)
      hipLaunchKernelGGL((k_level_scan<T, kScanChunkLevels>), glev, dim3(kScanThreads), tt * sizeof(float), st, nodes,
                         w.N, w.J, SZ);
    else
      hipLaunchKernelGGL((k_level_scan<T, kMaxLevels>), glev, dim3(kScanThreads), tt * sizeof(float), st, nodes, w.N,
                         w.J, SZ);
  }
  return launch_write_tag(a.workspace, w, mamba2_tag(a, sizeof(T), true), st);
}

// Enqueues the stages on `st`.  With `ev` non-null, ev[i] is recorded before stage i and ev[3]
// after the last one (used by the staged entry point): stage 0 block_state, stage 1 the level
// scan (lambda given) or the running scan (lambda == NULL), stage 2 tile_out.
template <typename T, int C, int DK, int DV>
hipError_t launch_mamba2(const Mamba2Args& a, hipStream_t st, hipEvent_t* ev) {
  constexpr int SZ = DK * DV;
  WsLayout w;
  mamba2_workspace(a.B, a.T, a.H, DK, DV, C, sizeof(T), a.lambda != nullptr, &w);
  const Nodes<T> nodes = mamba2_nodes<T>(w, a.workspace, a.lambda != nullptr);
  char* base = static_cast<char*>(a.workspace);
  T* tiles = nullptr;
  T* running = nullptr;
  if (!a.lambda) {
    tiles = reinterpret_cast<T*>(base + w.tiles);
    running = reinterpret_cast<T*>(base + w.running);
  }
  constexpr bool kFast = std::is_same<T, __bf16>::value && tile_rows(C) == kFastRows;
  const dim3 gtile((unsigned)(w.N * (kFast ? 1 : RowMap<tile_rows(C)>::RS) * a.H * a.B));
  if (ev) (void)hipEventRecord(ev[0], st);
  if (a.lambda) {
    const hipError_t e = launch_mamba2_summaries<T, C, DK, DV>(a, w, nodes, st, ev ? ev[1] : nullptr);
    if (e != hipSuccess) return e;
  } else {
    // the workspace no longer holds level summaries
    const hipError_t e = launch_write_tag(a.workspace, w, mamba2_tag(a, sizeof(T), false), st);
    if (e != hipSuccess) return e;
    const dim3 gblk((unsigned)(w.nb * a.H * a.B));
    const dim3 gscan((unsigned)((SZ / 2 + 255) / 256), (unsigned)(a.B * a.H));
    hipLaunchKernelGGL((k_block_state<T, C, DK, DV, false>), gblk, dim3(kStateThreads), 0, st, (const T*)a.k, (const T*)a.v,
                       a.log_alpha, nodes, tiles, const_cast<float*>(nodes.t1), a.T, (int)a.H, (int)a.Hqk);
    if (ev) (void)hipEventRecord(ev[1], st);
    hipLaunchKernelGGL((k_running_scan<T>), gscan, dim3(256), w.N * sizeof(float), st, (const T*)tiles, running,
                       (const float*)nodes.t1, w.N, SZ);
  }
  if (ev) (void)hipEventRecord(ev[2], st);
  if constexpr (kFast) {
    if (a.lambda)
      hipLaunchKernelGGL((k_tile_out_fast<DK, DV, true>), gtile, dim3(kFastThreads), 0, st, (const T*)a.q,
                         (const T*)a.k, (const T*)a.v, a.log_alpha, a.lambda, nodes, (const T*)running, (T*)a.o, a.T,
                         (int)a.H, (int)a.Hqk, a.L, w.J);
    else
      hipLaunchKernelGGL((k_tile_out_fast<DK, DV, false>), gtile, dim3(kFastThreads), 0, st, (const T*)a.q,
                         (const T*)a.k, (const T*)a.v, a.log_alpha, a.lambda, nodes, (const T*)running, (T*)a.o, a.T,
                         (int)a.H, (int)a.Hqk, a.L, w.J);
  } else {
    if (a.lambda)
      hipLaunchKernelGGL((k_tile_out<T, C, DK, DV, true>), gtile, dim3(RowMap<tile_rows(C)>::NT), 0, st, (const T*)a.q,
                         (const T*)a.k, (const T*)a.v, a.log_alpha, a.lambda, nodes, (const T*)running, (T*)a.o, a.T,
                         (int)a.H, (int)a.Hqk, a.L, w.J);
    else
      hipLaunchKernelGGL((k_tile_out<T, C, DK, DV, false>), gtile, dim3(RowMap<tile_rows(C)>::NT), 0, st, (const T*)a.q,
                         (const T*)a.k, (const T*)a.v, a.log_alpha, a.lambda, nodes, (const T*)running, (T*)a.o, a.T,
                         (int)a.H, (int)a.Hqk, a.L, w.J);
  }
  if (ev) (void)hipEventRecord(ev[3], st);
  return hipGetLastError();
}

int64_t mamba2_ml_workspace(int64_t B, int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t C, int64_t esize,
                            int L, bool full, int64_t* qlev_offset) {
  const int64_t fwd = mamba2_workspace(B, T, H, dk, dv, C, esize, true, nullptr);
  if (!full) return fwd;
  const int64_t base = (fwd + 255) & ~int64_t(255);
  if (qlev_offset) *qlev_offset = base;
  return base + B * T * H * L * dk * esize;
}

// Matrix-valued level weights: for full matrices the level queries go into the workspace (after
// the Fenwick summaries' regions) first; then the summaries and the tile outputs with per-level
// queries.  Events (optional, 5): before the level queries (an empty stage for diagonal weights),
// block_state, the level scan and tile_out, and after tile_out.
template <typename T, int C, int DK, int DV>
hipError_t launch_mamba2_ml(const Mamba2Args& a, hipStream_t st, hipEvent_t* ev) {
  WsLayout w;
  mamba2_workspace(a.B, a.T, a.H, DK, DV, C, sizeof(T), true, &w);
  int64_t qoff = 0;
  mamba2_ml_workspace(a.B, a.T, a.H, DK, DV, C, sizeof(T), a.L, a.lambda_full, &qoff);
  const Nodes<T> nodes = mamba2_nodes<T>(w, a.workspace, true);
  T* qlev = reinterpret_cast<T*>(static_cast<char*>(a.workspace) + qoff);
  const int64_t rows = a.B * a.T * a.H;
  if (ev) (void)hipEventRecord(ev[0], st);
  if (a.lambda_full) {
    const int64_t nblk = (rows * a.L + kLevelQueryThreads / 64 - 1) / (kLevelQueryThreads / 64);
    hipLaunchKernelGGL((k_level_queries_full<T, DK>), dim3((unsigned)nblk), dim3(kLevelQueryThreads), 0, st,
                       (const T*)a.q, a.lambda_matrix, qlev, rows, a.L);
  }
  if (ev) (void)hipEventRecord(ev[1], st);
  hipError_t e = launch_mamba2_summaries<T, C, DK, DV>(a, w, nodes, st, ev ? ev[2] : nullptr);
  if (e != hipSuccess) return e;
  if (ev) (void)hipEventRecord(ev[3], st);
  const dim3 gtile((unsigned)(w.N * RowMap<tile_rows(C)>::RS * a.H * a.B));
  if (a.lambda_full)
    hipLaunchKernelGGL((k_tile_out<T, C, DK, DV, true, 1>), gtile, dim3(RowMap<tile_rows(C)>::NT), 0, st,
                       (const T*)qlev, (const T*)a.k, (const T*)a.v, a.log_alpha, (const float*)nullptr, nodes,
                       (const T*)nullptr, (T*)a.o, a.T, (int)a.H, (int)a.H, a.L, w.J);
  else
    hipLaunchKernelGGL((k_tile_out<T, C, DK, DV, true, 2>), gtile, dim3(RowMap<tile_rows(C)>::NT), 0, st,
                       (const T*)a.q, (const T*)a.k, (const T*)a.v, a.log_alpha, a.lambda_matrix, nodes,
                       (const T*)nullptr, (T*)a.o, a.T, (int)a.H, (int)a.H, a.L, w.J);
  if (ev) (void)hipEventRecord(ev[4], st);
  return hipGetLastError();
}

hipError_t launch_debug_level_map(int64_t T, int64_t C, int8_t* out, hipStream_t st) {
  const int R = tile_rows((int)C);
  hipLaunchKernelGGL(k_debug_level_map, dim3((unsigned)T), dim3(256), 0, st, T, R, bitlen_h(uint64_t(R)) - 1,
                     tile_levels(T, C), out);
  return hipGetLastError();
}

#define LL_SUMMARIES_INST(T, C, DK, DV)                                                                     \
  template hipError_t launch_mamba2_summaries<T, C, DK, DV>(const Mamba2Args&, const WsLayout&, const Nodes<T>&, \
                                                            hipStream_t, hipEvent_t);
LL_MAMBA2_SHAPES(LL_SUMMARIES_INST)
#undef LL_SUMMARIES_INST

const KernelEntry* mamba2_table(int* n) {
#define LL_ENTRY(T, C, DK, DV) \
  {std::is_same<T, float>::value ? 0 : 1, C, DK, DV, &launch_mamba2<T, C, DK, DV>, &launch_mamba2_ml<T, C, DK, DV>},
  static const KernelEntry table[] = {LL_MAMBA2_SHAPES(LL_ENTRY)};
#undef LL_ENTRY
  *n = sizeof(table) / sizeof(table[0]);
  return table;
}

}  // namespace ll
