// Log-linear Gated DeltaNet forward (Sec. 3.4): O = (A (.) M^S (.) M^H) V with
// A = (Q K^T (.) L)(I + diag(beta)(K K^T (.) (L - I)))^{-1} diag(beta), i.e. the recurrence
// S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T read out per Fenwick level.
//
// Chunkwise form (chunks of C tokens; local rows t, s; gamma_t = exp(cl_t) with cl the
// chunk-local inclusive cumulative log-gate; Gamma[t,s] = gamma_t / gamma_s for s <= t):
//   T_G   = (I + diag(beta)(K K^T (.) Gamma (.) (L - I)))^{-1} diag(beta)   (unit-lower solve)
//   W     = T_G diag(gamma) K,   U = T_G V                                   (WY / UT form)
//   P_G   = Q K^T (.) Gamma (.) L
//   intra : O_c = ((P_G T_G) (.) M^H_c) V       -- the chunk's own block of A, level-masked
//   Qc    = diag(gamma) Q - P_G W               -- query seen through the chunk's transitions
//   state : S_end^T = P_z S_start^T + H_z,  P_z = gamma_C I - K~^T W,  H_z = K~^T U,
//           K~ = diag(exp(tot - cl)) K
// An earlier state S (d_v x d_k) reaches row t of the chunk as S q~_t (q~_t = row t of Qc).
// Inter-chunk levels (Sec. 3.3 with the delta-rule transition): per chunk level j the state
// R_j (d_k x d_v) restarts at every chunk z with z % 2^j == 0, absorbs H_z in the source half
// (bit j-1 of z clear) and propagates through P_z everywhere; a chunk with bit j-1 set adds
// lambda_t^(log2 C + j) q~_t^T R_j to its rows, with R_j taken at the chunk's start.
//
// Block tree instead of a sequential scan.  For a block of chunks [a, c) let T = P_{c-1} ... P_a
// (its transition) and A = sum over s in [a, c) of P_{c-1} ... P_{s+1} H_s (its accumulated state);
// the block [a, c) = [a, b) then [b, c) has T = T_hi T_lo and A = T_hi A_lo + A_hi.  The level-j
// state read by chunk z (bit j-1 set) is R_j = T(G_1) ... T(G_{j-1}) A(G_j), with G_j the aligned
// source group of 2^(j-1) chunks ending at ((z >> (j-1)) << (j-1)) and G_1, .. the lower source
// groups of z (its set bits below j-1), the most recent first.  So a chunk reads its levels from
// the lowest set bit up, carrying q~^T through each group's transition: out += lambda^(j) q~^T A(G_j),
// then q~^T <- q~^T T(G_j).  Every source group is the aligned block (level j-1, index
// (z >> (j-1)) - 1) of a binary block tree built level by level.
//
// Kernels: gdn_chunk (one persistent workgroup per compute unit walking its chunks; per chunk the WY
// solve in fp32 by a blocked inversion and all chunk-local products on MFMA, bf16 operands with fp32
// accumulation), gdn_combine (one launch per tree level, one workgroup per block) and gdn_read (one
// workgroup per chunk: the level read-out and the final output).
#include <type_traits>

#include "ll_device.hpp"
#include "ll_launch.hpp"

namespace ll {

namespace gdn {

constexpr int kMaxJ = 16;      // inter-chunk levels handled by the read-out (T <= C * 2^16)
constexpr int kChunkWaves = 8; // waves per gdn_chunk workgroup
typedef __bf16 bf;

// Element offset of entry (r, k) of a staged bf16 matrix with rows of ld elements whose 8-element
// chunks are XOR-swizzled by row group when SW: chunk k / 8 of row r sits at position
// (k / 8) ^ ((r / 8) % 8).  Used for the transposed (d-major) copies of the chunk's K and V, whose
// rows of C = 64 tokens are written eight rows at a time (see the staging in k_gdn_chunk).
template <bool SW>
__device__ inline int stg(int r, int ld, int k) {
  return r * ld + (SW ? ((((k >> 3) ^ (r >> 3)) & 7) << 3) + (k & 7) : k);
}

// C = A B over 16x16 output tiles, A [M][K] row-major (lda), Bt = B^T [N][K] row-major (ldb), both
// bf16 in LDS (SWA / SWB: the operand's chunks are swizzled as by stg, K = 64); tiles dealt
// round-robin to the kChunkWaves waves; epi(mt, nt, acc) consumes each tile (lane holds column
// 16 nt + (lane & 15), rows 16 mt + 4 (lane >> 4) + r).
template <int M, int N, int K, bool SWA = false, bool SWB = false, typename Epi>
__device__ inline void gemm_lds(const bf* A, int lda, const bf* Bt, int ldb, Epi epi) {
  using MF = Mfma<bf>;
  static_assert(!(SWA || SWB) || K == 64, "swizzled operands have rows of 64 elements");
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, r16 = lane & 15, g = lane >> 4;
  constexpr int MT = M / 16, NT = N / 16;
  for (int tile = wave; tile < MT * NT; tile += kChunkWaves) {
    const int mt = tile / NT, nt = tile % NT;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < K / MF::KSTEP; ++ks) {
      const int k0 = ks * MF::KSTEP + g * MF::KPL;
      acc = MF::mma(MF::load(&A[stg<SWA>(mt * 16 + r16, lda, k0)]), MF::load(&Bt[stg<SWB>(nt * 16 + r16, ldb, k0)]), acc);
    }
    epi(mt, nt, acc);
  }
}

// As gemm_lds with the wave's tiles unrolled: epi(i, mt, nt, acc) for the wave's i-th tile
// (tile wave + kChunkWaves i), so that the epilogue can index registers by i.
template <int M, int N, int K, typename Epi>
__device__ inline void gemm_lds_unrolled(const bf* A, int lda, const bf* Bt, int ldb, Epi epi) {
  using MF = Mfma<bf>;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, r16 = lane & 15, g = lane >> 4;
  constexpr int MT = M / 16, NT = N / 16;
  static_assert(MT * NT % kChunkWaves == 0, "whole rounds of tiles");
#pragma unroll
  for (int i = 0; i < MT * NT / kChunkWaves; ++i) {
    const int tile = wave + i * kChunkWaves, mt = tile / NT, nt = tile % NT;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < K / MF::KSTEP; ++ks) {
      const int k0 = ks * MF::KSTEP + g * MF::KPL;
      acc = MF::mma(MF::load(&A[(mt * 16 + r16) * lda + k0]), MF::load(&Bt[(nt * 16 + r16) * ldb + k0]), acc);
    }
    epi(i, mt, nt, acc);
  }
}

// "kfrag" layout of a K x N bf16 matrix X (KR = K rows), in which X is read as the B operand of a
// product Y X: the operand fragment of column tile nt and k step ks (32 rows) is 64 lanes x 8
// elements, lane (n % 16) + 16 ((k % 32) / 8) holding rows k with k % 8 = 0..7 in order.  The same
// bytes are the A-operand fragments of X^T (row tile nt of X^T, k step ks).  Four consecutive rows
// 4i .. 4i + 3 of one column are four consecutive elements.
template <int KR>
__device__ inline int kfrag_idx(int k, int n) {
  return (((n >> 4) * (KR / 32) + (k >> 5)) * 64 + (n & 15) + 16 * ((k & 31) >> 3)) * 8 + (k & 7);
}

// ---------------------------------------------------------------------------------------------
// Kernel 1: per-chunk WY solve and chunk-local products.  One workgroup (kChunkWaves waves) per chunk.
// Outputs (workspace, per chunk): Qc [C][DK] bf16 row-major, P_z [DK][DK] bf16 (kfrag layout for
// even chunks z, row-major for odd ones: the two sides of a tree combination), H_z [DK][DV] bf16
// (kfrag), intra-chunk output [C][DV] fp32 in the MFMA result layout (16 x 16 tiles, row tile
// major; lane l of a tile holds rows 4 (l / 16) + 0..3 of column l % 16).
// ---------------------------------------------------------------------------------------------
template <int C, int DK, int DV, bool HAS_LAMBDA>
__global__ __launch_bounds__(64 * kChunkWaves) void k_gdn_chunk(const bf* __restrict__ q, const bf* __restrict__ k,
                                                   const bf* __restrict__ v, const float* __restrict__ log_alpha,
                                                   const float* __restrict__ beta, const float* __restrict__ lam,
                                                   bf* __restrict__ qc_out, bf* __restrict__ pz_out,
                                                   bf* __restrict__ hz_out, float* __restrict__ oin_out,
                                                   int64_t Tlen, int H, int L, int64_t nchunks) {
  static_assert(C == 64, "the inversion works on 4 x 4 blocks of 16 x 16 (one lane per column of wave 0)");
  constexpr int LOG2C = 6;
  constexpr int PD = 8;                 // row padding (elements)
  constexpr int LDD = DK + PD;          // rows of length d_k
  constexpr int LDC = C + PD;           // rows of length C
  constexpr int VEC = 8;
  constexpr int LDL = C + 4;            // fp32 L rows: 16-byte aligned, read four entries at a time
  // region 1: phase A/B (K, Q row-major, fp32 L) reused in phase C/D (W^T, U^T, masked P)
  constexpr int R1A = 2 * C * LDD * 2 + C * LDL * 4;
  constexpr int R1B = (DK * LDC + DV * LDC + C * LDC) * 2;
  constexpr int R1 = R1A > R1B ? R1A : R1B;
  __shared__ __attribute__((aligned(16))) char r1[R1];
  __shared__ bf kgt_s[DK * LDC];   // (gamma K)^T, chunks swizzled (stg)
  __shared__ bf kdt_s[DK * LDC];   // (decay-to-end K)^T, chunks swizzled
  __shared__ bf vt_s[DV * LDC];    // V^T, chunks swizzled
  __shared__ bf pg_s[C * LDC];     // P_G
  __shared__ bf z_s[C * LDC];      // T_G
  __shared__ bf zt_s[C * LDC];     // T_G^T
  __shared__ float cl_s[C], gm_s[C], dc_s[C], bt_s[C];
  __shared__ float lam_s[HAS_LAMBDA ? C * (LOG2C + 1) : 1];
  __shared__ float xs_s[10 * 256];  // fp32 blocks (i, j), j <= i, of X = (I + L)^{-1}: block i(i+1)/2 + j
  bf* k_s = reinterpret_cast<bf*>(r1);
  bf* q_s = k_s + C * LDD;
  float* l_s = reinterpret_cast<float*>(r1 + 2 * C * LDD * 2);
  bf* wt_s = reinterpret_cast<bf*>(r1);
  bf* ut_s = wt_s + DK * LDC;
  bf* ph_s = ut_s + DV * LDC;

  const int64_t N = Tlen / C;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, r16 = lane & 15, g = lane >> 4;

  // A persistent grid: the workgroup takes chunks blockIdx.x, blockIdx.x + gridDim.x, ... (logical
  // order (b, h, z) through the XCD mapping), and loads the next chunk's inputs (K, Q, V rows, gates,
  // beta, lambda) into registers as soon as the current chunk has staged its own, so that their
  // memory latency overlaps the current chunk's work.  A wave instruction loads 16-byte pieces of
  // 8 tokens x 8 consecutive pieces (piece p of the tensor: token 8 (b % 8) + (l % 8), columns
  // 8 (8 (b / 8) + l / 8) .. + 7, with b = p / 64 and l = p % 64): whole 128-byte lines, and in the
  // transposed LDS copies eight rows 8 apart whose swizzled chunks fall in distinct banks.
  constexpr int NTH = 64 * kChunkWaves;
  constexpr int NKQ = C * DK / VEC / NTH, NVV = C * DV / VEC / NTH;  // 16-byte pieces per thread
  static_assert(C == 64, "pieces of 8 tokens x 8 column pieces");
  auto piece_t = [&](int p) { return ((p >> 6) & 7) * 8 + (p & 7); };        // token of piece p
  auto piece_d = [&](int p) { return (((p >> 6) >> 3) * 8 + ((p & 63) >> 3)) * VEC; };  // first column
  constexpr int NLW = HAS_LAMBDA ? (C * (LOG2C + 1) + NTH - 1) / NTH : 1;  // lambda values per thread
  static_assert(C * DK / VEC % NTH == 0 && C * DV / VEC % NTH == 0, "whole passes of the workgroup");
  bf16x8 kpre[NKQ], qpre[NKQ], vpre[NVV];
  float la_r = 0.f, bt_r = 0.f, lam_r[NLW];
  auto load_inputs = [&](int64_t it) {
    const int64_t wk = xcd_remap(it, nchunks);
    const int64_t zz = wk % N, bhh = wk / N;
    const int hh = (int)(bhh % H), bb = (int)(bhh / H);
    const int64_t t0 = (int64_t)bb * Tlen + zz * C;
    // the small loads first and unconditionally (every wave, clamped indices; only wave 0 and the
    // in-range entries are used), so that no wave waits on them where their registers are reused
    la_r = log_alpha[(t0 + lane) * H + hh];  // scaled at its use: nothing waits for the load here
    bt_r = beta[(t0 + lane) * H + hh];
    if constexpr (HAS_LAMBDA) {
#pragma unroll
      for (int e = 0; e < NLW; ++e) {
        const int idx = tid + e * NTH, ic = idx < C * (LOG2C + 1) ? idx : C * (LOG2C + 1) - 1;
        lam_r[e] = lam[((t0 + ic / (LOG2C + 1)) * H + hh) * L + ic % (LOG2C + 1)];
      }
    }
#pragma unroll
    for (int e = 0; e < NKQ; ++e) {
      const int idx = tid + e * NTH, t = piece_t(idx), d0 = piece_d(idx);
      kpre[e] = *reinterpret_cast<const bf16x8*>(k + ((t0 + t) * H + hh) * DK + d0);
    }
  };
  // Q is prefetched in phase C
  auto load_q = [&](int64_t it) {
    const int64_t wk = xcd_remap(it, nchunks);
    const int64_t zz = wk % N, bhh = wk / N;
    const int hh = (int)(bhh % H), bb = (int)(bhh / H);
    const int64_t t0 = (int64_t)bb * Tlen + zz * C;
#pragma unroll
    for (int e = 0; e < NKQ; ++e) {
      const int idx = tid + e * NTH, t = piece_t(idx), d0 = piece_d(idx);
      qpre[e] = *reinterpret_cast<const bf16x8*>(q + ((t0 + t) * H + hh) * DK + d0);
    }
  };
  // V is prefetched separately, later in the chunk (phase B), so that no wave issues the whole
  // burst at once
  auto load_v = [&](int64_t it) {
    const int64_t wk = xcd_remap(it, nchunks);
    const int64_t zz = wk % N, bhh = wk / N;
    const int hh = (int)(bhh % H), bb = (int)(bhh / H);
    const int64_t t0 = (int64_t)bb * Tlen + zz * C;
#pragma unroll
    for (int e = 0; e < NVV; ++e) {
      const int idx = tid + e * NTH, t = piece_t(idx), d0 = piece_d(idx);
      vpre[e] = *reinterpret_cast<const bf16x8*>(v + ((t0 + t) * H + hh) * DV + d0);
    }
  };
  if (blockIdx.x < nchunks) {
    load_inputs(blockIdx.x);
    load_v(blockIdx.x);
    load_q(blockIdx.x);
  }
  // The first chunk's inputs are awaited here, once: the compiler's counter waits at the loop head
  // then see, on every path into it, the epilogue stores issued after the prefetch, and no longer
  // wait for those stores to drain before each chunk's first use of its prefetched inputs.
  wait_vmem();
  for (int64_t it = blockIdx.x; it < nchunks; it += gridDim.x) {
  const int64_t work = xcd_remap(it, nchunks);  // (b, h, z)
  const int64_t z = work % N;
  const int64_t bh = work / N;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int64_t tok0 = (int64_t)b * Tlen + z * C;
  const int64_t cidx = bh * N + z;
  __syncthreads();  // the previous chunk's readers of LDS are done

  // ---- phase A: gates, staging, K K^T and Q K^T
  if (wave == 0) {
    const float la = lane < C ? la_r * kLog2e : 0.f;
    const float cl = wave_inclusive_scan(la);
    const float tot = __shfl(cl, C - 1, 64);
    if (lane < C) {
      cl_s[lane] = cl;
      gm_s[lane] = fast_exp2(cl);
      dc_s[lane] = fast_exp2(tot - cl);
      bt_s[lane] = bt_r;
    }
  }
  if constexpr (HAS_LAMBDA) {
#pragma unroll
    for (int e = 0; e < NLW; ++e) {
      const int idx = tid + e * NTH;
      if (idx < C * (LOG2C + 1)) lam_s[idx] = lam_r[e];
    }
  }
  __syncthreads();
#pragma unroll
  for (int e = 0; e < NKQ; ++e) {
    const int idx = tid + e * NTH, t = piece_t(idx), d0 = piece_d(idx);
    const bf16x8 kv = kpre[e], qv = qpre[e];
    *reinterpret_cast<bf16x8*>(&k_s[t * LDD + d0]) = kv;
    *reinterpret_cast<bf16x8*>(&q_s[t * LDD + d0]) = qv;
    const float gt = gm_s[t], dt = dc_s[t];
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const float x = static_cast<float>(kv[e]);
      kgt_s[stg<true>(d0 + e, LDC, t)] = static_cast<bf>(x * gt);
      kdt_s[stg<true>(d0 + e, LDC, t)] = static_cast<bf>(x * dt);
    }
  }
#pragma unroll
  for (int e = 0; e < NVV; ++e) {
    const int idx = tid + e * NTH, t = piece_t(idx), d0 = piece_d(idx);
    const bf16x8 vv = vpre[e];
#pragma unroll
    for (int e = 0; e < VEC; ++e) vt_s[stg<true>(d0 + e, LDC, t)] = vv[e];
  }
  if (it + gridDim.x < nchunks) load_inputs(it + gridDim.x);  // the next chunk's, while this one runs
  __syncthreads();
  // the Q entries of this lane's tiles of the corrected-query product (formed transposed: tile
  // (mt, nt) holds columns d = 16 mt + 4 g + 0..3 of row t = 16 nt + (lane & 15)), read while Q is
  // staged (its LDS region is reused by phase C), so that the product's epilogue issues no loads
  constexpr int QCT = (DK / 16) * (C / 16) / kChunkWaves;
  bf16x4 qreg[QCT];
#pragma unroll
  for (int i = 0; i < QCT; ++i) {
    const int tile = wave + i * kChunkWaves, mt = tile / (C / 16), nt = tile % (C / 16);
    qreg[i] = *reinterpret_cast<const bf16x4*>(&q_s[(nt * 16 + r16) * LDD + mt * 16 + 4 * g]);
  }
  // L[t][s] = beta_t (k_t . k_s) Gamma[t,s] for s < t (fp32);  P_G[t][s] = (q_t . k_s) Gamma[t,s], s <= t
  gemm_lds<C, C, DK>(k_s, LDD, k_s, LDD, [&](int mt, int nt, f32x4 acc) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = mt * 16 + 4 * g + r, s = nt * 16 + r16;
      l_s[t * LDL + s] = s < t ? bt_s[t] * acc[r] * fast_exp2(cl_s[t] - cl_s[s]) : 0.f;
    }
  });
  __syncthreads();

  // ---- phase B: X = (I + L)^{-1} in 16 x 16 blocks (fp32), T_G = X diag(beta) into z_s[t][c] and
  //      zt_s[c][t].  B1: wave 0 inverts the four diagonal blocks by forward substitution (lane
  //      16 b + c = column c of block b) while the other waves form P_G and zero the blocks above
  //      the diagonal.  B2: block row i = 1, 2, 3 in turn, X_ij = -X_ii sum_{k=j}^{i-1} L_ik X_kj,
  //      tile (i, j) on wave j (fp32 MFMA).
  auto blk = [](int i, int j) { return (i * (i + 1) / 2 + j) * 256; };
  auto put_t = [&](int t, int c, float x) {  // T_G entry (t, c)
    const bf zv = static_cast<bf>(x * bt_s[c]);
    z_s[t * LDC + c] = zv;
    zt_s[c * LDC + t] = zv;
  };
  const bool more = it + gridDim.x < nchunks;
  if (wave != 0) {
    if (more) load_v(it + gridDim.x);
    // P_G[t][s] = (q_t . k_s) Gamma[t,s], s <= t, 16 x 16 tiles dealt to the other waves
    using MF = Mfma<bf>;
    constexpr int MT = C / 16;
    for (int tile = wave - 1; tile < MT * MT; tile += kChunkWaves - 1) {
      const int mt = tile / MT, nt = tile % MT;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < DK / MF::KSTEP; ++ks) {
        const int k0 = ks * MF::KSTEP + g * MF::KPL;
        acc = MF::mma(MF::load(&q_s[(mt * 16 + r16) * LDD + k0]), MF::load(&k_s[(nt * 16 + r16) * LDD + k0]), acc);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = mt * 16 + 4 * g + r, s = nt * 16 + r16;
        pg_s[t * LDC + s] = static_cast<bf>(s <= t ? acc[r] * fast_exp2(cl_s[t] - cl_s[s]) : 0.f);
      }
    }
    // zeros above the diagonal blocks (rows of block i, columns of block j > i)
    for (int idx = tid - 64; idx < 6 * 256; idx += 64 * (kChunkWaves - 1)) {
      const int bj = idx >> 8, e = idx & 255;
      const int bi = bj < 3 ? 0 : (bj < 5 ? 1 : 2);                // (0,1) (0,2) (0,3) (1,2) (1,3) (2,3)
      const int bc = bj < 3 ? bj + 1 : (bj < 5 ? bj - 1 : 3);
      const int t = 16 * bi + (e >> 4), c = 16 * bc + (e & 15);
      z_s[t * LDC + c] = static_cast<bf>(0.f);
      zt_s[c * LDC + t] = static_cast<bf>(0.f);
    }
  } else {
    const int bb = lane >> 4, c = lane & 15;
    const float* lb = l_s + 16 * bb * LDL + 16 * bb;  // diagonal block bb of L
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
      for (int j = 0; j + 3 < i; j += 4) {
        const f32x4 lv = *reinterpret_cast<const f32x4*>(&lb[i * LDL + j]);  // broadcast per block
        a0 += lv[0] * x[j];
        a1 += lv[1] * x[j + 1];
        a2 += lv[2] * x[j + 2];
        a3 += lv[3] * x[j + 3];
      }
#pragma unroll
      for (int j = i & ~3; j < i; ++j) a0 += lb[i * LDL + j] * x[j];
      const float acc = ((i == c) ? 1.f : 0.f) - ((a0 + a1) + (a2 + a3));
      x[i] = (i < c) ? 0.f : acc;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      xs_s[blk(bb, bb) + i * 16 + c] = x[i];
      put_t(16 * bb + i, 16 * bb + c, x[i]);
    }
    if (more) load_v(it + gridDim.x);
  }
  for (int i = 1; i < C / 16; ++i) {
    __syncthreads();  // blocks of rows < i (and the diagonal ones) are in xs_s
    if (wave < i) {
      using MF = Mfma<float>;
      const int jb = wave;
      // Y = sum_{k=j}^{i-1} L_ik X_kj  (k slot 4 kk + g)
      f32x4 y = {0.f, 0.f, 0.f, 0.f};
      for (int kb = jb; kb < i; ++kb) {
        const float* xb = xs_s + blk(kb, jb);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          y = MF::mma(l_s[(16 * i + r16) * LDL + 16 * kb + 4 * kk + g], xb[(4 * kk + g) * 16 + r16], y);
      }
      // X_ij = -X_ii Y  (k slot 4 g + r: Y in the result layout is the B operand directly)
      const float* di = xs_s + blk(i, i);
      f32x4 xv = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int r = 0; r < 4; ++r) xv = MF::mma(di[r16 * 16 + 4 * g + r], y[r], xv);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float xr = -xv[r];
        xs_s[blk(i, jb) + (4 * g + r) * 16 + r16] = xr;
        put_t(16 * i + 4 * g + r, 16 * jb + r16, xr);
      }
    }
  }
  __syncthreads();

  // ---- phase C: W = T_G (gamma K), U = T_G V (stored transposed), A_c = P_G T_G masked by M^H
  if (more) load_q(it + gridDim.x);
  gemm_lds<C, DK, C, false, true>(z_s, LDC, kgt_s, LDC, [&](int mt, int nt, f32x4 acc) {
    bf16x4 w4;
#pragma unroll
    for (int r = 0; r < 4; ++r) w4[r] = static_cast<bf>(acc[r]);
    *reinterpret_cast<bf16x4*>(&wt_s[(nt * 16 + r16) * LDC + mt * 16 + 4 * g]) = w4;
  });
  gemm_lds<C, DV, C, false, true>(z_s, LDC, vt_s, LDC, [&](int mt, int nt, f32x4 acc) {
    bf16x4 u4;
#pragma unroll
    for (int r = 0; r < 4; ++r) u4[r] = static_cast<bf>(acc[r]);
    *reinterpret_cast<bf16x4*>(&ut_s[(nt * 16 + r16) * LDC + mt * 16 + 4 * g]) = u4;
  });
  gemm_lds<C, C, C>(pg_s, LDC, zt_s, LDC, [&](int mt, int nt, f32x4 acc) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = mt * 16 + 4 * g + r, s = nt * 16 + r16;
      float w = s <= t ? acc[r] : 0.f;
      if constexpr (HAS_LAMBDA) w *= lam_s[t * (LOG2C + 1) + level_local(t, s)];
      ph_s[t * LDC + s] = static_cast<bf>(w);
    }
  });
  __syncthreads();

  // ---- phase D: intra output, corrected queries, transition and chunk state
  // the intra output in the MFMA result layout, tile by tile (one 1 KB store per tile; the
  // read-out kernel adds it to accumulators of the same layout)
  float* oin = oin_out + cidx * (C * DV);
  gemm_lds<C, DV, C, false, true>(ph_s, LDC, vt_s, LDC, [&](int mt, int nt, f32x4 acc) {
    *reinterpret_cast<f32x4*>(oin + ((mt * (DV / 16) + nt) * 64 + lane) * 4) = acc;
  });
  bf* qc = qc_out + cidx * (C * DK);
  // Qc^T = gamma Q^T - W^T P_G^T: four consecutive columns of one row of Qc per lane, one 8-byte
  // store each
  gemm_lds_unrolled<DK, C, C>(wt_s, LDC, pg_s, LDC, [&](int i, int mt, int nt, f32x4 acc) {
    const int d0 = mt * 16 + 4 * g, t = nt * 16 + r16;
    const float gt = gm_s[t];
    bf16x4 q4;
#pragma unroll
    for (int r = 0; r < 4; ++r) q4[r] = static_cast<bf>(gt * static_cast<float>(qreg[i][r]) - acc[r]);
    *reinterpret_cast<bf16x4*>(qc + t * DK + d0) = q4;
  });
  bf* pz = pz_out + cidx * (DK * DK);
  const float gC = gm_s[C - 1];
  // P_z = gamma_C I - K~^T W, stored four consecutive elements per lane: an even chunk's in the
  // kfrag layout (rows d .. d + 3 of column e), an odd chunk's row-major from the transposed
  // product (columns e .. e + 3 of row d)
  if (!(z & 1)) {
    gemm_lds<DK, DK, C, true, false>(kdt_s, LDC, wt_s, LDC, [&](int mt, int nt, f32x4 acc) {
      const int d0 = mt * 16 + 4 * g, e = nt * 16 + r16;
      bf16x4 p4;
#pragma unroll
      for (int r = 0; r < 4; ++r) p4[r] = static_cast<bf>((d0 + r == e ? gC : 0.f) - acc[r]);
      *reinterpret_cast<bf16x4*>(pz + kfrag_idx<DK>(d0, e)) = p4;
    });
  } else {
    gemm_lds<DK, DK, C, false, true>(wt_s, LDC, kdt_s, LDC, [&](int mt, int nt, f32x4 acc) {
      const int e0 = mt * 16 + 4 * g, d = nt * 16 + r16;
      bf16x4 p4;
#pragma unroll
      for (int r = 0; r < 4; ++r) p4[r] = static_cast<bf>((d == e0 + r ? gC : 0.f) - acc[r]);
      *reinterpret_cast<bf16x4*>(pz + d * DK + e0) = p4;
    });
  }
  bf* hz = hz_out + cidx * (DK * DV);
  gemm_lds<DK, DV, C, true, false>(kdt_s, LDC, ut_s, LDC, [&](int mt, int nt, f32x4 acc) {
    bf16x4 h4;
#pragma unroll
    for (int r = 0; r < 4; ++r) h4[r] = static_cast<bf>(acc[r]);
    *reinterpret_cast<bf16x4*>(hz + kfrag_idx<DK>(mt * 16 + 4 * g, nt * 16 + r16)) = h4;
  });
  }  // chunk loop
}

// ---------------------------------------------------------------------------------------------
// Kernel 2: one level m >= 1 of the block tree.  Block (m, k) of a sequence covers chunks
// [k 2^m, (k + 1) 2^m).  It is formed from blocks lo = 2k and hi = 2k + 1 of level m - 1:
// T = T_hi T_lo, A = T_hi A_lo + A_hi, fp32 accumulation, one RNE cast.  Storage of a block:
// T (DK x DK) then A (DK x DV), A in the kfrag layout, T in the kfrag layout when k is even (the
// source groups that chunks read, and the lo side of the next level) and row-major when k is odd
// (the hi side).  Level 0 is the chunk kernel's P_z and H_z (same layout rule, by chunk parity).
// The (DK + DV) / 16 column tiles of [T | A] are split over workgroups of kCombineTiles column
// tiles, which the dispatch-order remap keeps on one XCD; wave w forms rows 16 (RT w + i) + 0..15
// of its workgroup's tiles (RT = DK / 64).  An odd block's T is formed transposed
// (T^T = T_lo^T T_hi^T) so that its rows are stored whole.  Every operand fragment of a workgroup
// is loaded up front; the B-operand fragments, the same for every wave, go through LDS.
// ---------------------------------------------------------------------------------------------
constexpr int kCombineTiles = 4;  // column tiles per workgroup

template <int DK, int DV>
__global__ __launch_bounds__(256) void k_gdn_combine(const bf* __restrict__ t_in, const bf* __restrict__ a_in,
                                                     int64_t t_stride, int64_t a_stride, int64_t n_in,
                                                     bf* __restrict__ out, int64_t n_out) {
  using MF = Mfma<bf>;
  typedef MF::frag frag;
  constexpr int KS = DK / 32, RT = DK / 64;  // k steps; row tiles per wave
  constexpr int TT = DK / 16, AT = DV / 16;  // column tiles of T and A
  constexpr int CT = kCombineTiles, S = (TT + AT) / CT;
  static_assert(TT % CT == 0 && AT % CT == 0, "a workgroup's tiles lie in T or in A");
  static_assert(CT * KS % 4 == 0, "the B fragments split evenly over the four waves");
  constexpr int BS = DK * (DK + DV);
  const int64_t id = xcd_remap(blockIdx.x, (int64_t)gridDim.x);
  const int64_t kb = id / S, bh = blockIdx.y;
  const int c0 = (int)(id % S) * CT;  // first column tile of [T | A]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, r16 = lane & 15, g = lane >> 4;
  const bf* tlo = t_in + (bh * n_in + 2 * kb) * t_stride;
  const bf* thi = tlo + t_stride;
  const bf* alo = a_in + (bh * n_in + 2 * kb) * a_stride;
  const bf* ahi = alo + a_stride;
  bf* tout = out + (bh * n_out + kb) * BS;
  bf* aout = tout + DK * DK;
  const bool t_part = c0 < TT, transposed = t_part && (kb & 1);

  // A operand: rows of T_hi (row-major), or for a transposed T the rows of T_lo^T (kfrag of T_lo);
  // rows 16 (RT wave + i) + r16, k = 32 ks + 8 g + 0..7
  frag fa[RT][KS];
  // B operand of column tile c0 + c: A_lo or T_lo (kfrag), or for a transposed T the rows of T_hi.
  // The same for every wave: each wave loads a quarter of them into LDS and reads all back.
  __shared__ frag fb_s[CT * KS][64];
  constexpr int FPW = CT * KS / 4;  // B fragments loaded per wave
  frag fbw[FPW];
#pragma unroll
  for (int x = 0; x < FPW; ++x) {
    const int f = wave + 4 * x, c = f / KS, ks = f % KS;
    const int nt = t_part ? c0 + c : c0 - TT + c;
    fbw[x] = transposed ? MF::load(thi + (16 * nt + r16) * DK + 32 * ks + 8 * g)
                        : MF::load((t_part ? tlo : alo) + ((nt * KS + ks) * 64 + lane) * 8);
  }
#pragma unroll
  for (int i = 0; i < RT; ++i)
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      fa[i][ks] = transposed ? MF::load(tlo + (((RT * wave + i) * KS + ks) * 64 + lane) * 8)
                             : MF::load(thi + (16 * (RT * wave + i) + r16) * DK + 32 * ks + 8 * g);
  // A_hi (added to the A tiles) with the operands, not after the products
  bf16x4 ahv[CT][RT];
  if (!t_part) {
#pragma unroll
    for (int c = 0; c < CT; ++c)
#pragma unroll
      for (int i = 0; i < RT; ++i)
        ahv[c][i] = *reinterpret_cast<const bf16x4*>(ahi + kfrag_idx<DK>(16 * (RT * wave + i) + 4 * g, 16 * (c0 - TT + c) + r16));
  }
#pragma unroll
  for (int x = 0; x < FPW; ++x) fb_s[wave + 4 * x][lane] = fbw[x];
  __syncthreads();
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    const int nt = t_part ? c0 + c : c0 - TT + c;
    f32x4 acc[RT];
#pragma unroll
    for (int i = 0; i < RT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int i = 0; i < RT; ++i) acc[i] = MF::mma(fa[i][ks], fb_s[c * KS + ks][lane], acc[i]);
#pragma unroll
    for (int i = 0; i < RT; ++i) {
      const int row0 = 16 * (RT * wave + i) + 4 * g;
      bf16x4 res;
      if (!t_part) {  // A = T_hi A_lo + A_hi; the lane's four rows are four consecutive kfrag elements
        const int idx = kfrag_idx<DK>(row0, 16 * nt + r16);
        const bf16x4 add = ahv[c][i];
#pragma unroll
        for (int r = 0; r < 4; ++r) res[r] = static_cast<bf>(acc[i][r] + static_cast<float>(add[r]));
        *reinterpret_cast<bf16x4*>(aout + idx) = res;
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) res[r] = static_cast<bf>(acc[i][r]);
        if (!transposed)  // T = T_hi T_lo, kfrag
          *reinterpret_cast<bf16x4*>(tout + kfrag_idx<DK>(row0, 16 * nt + r16)) = res;
        else  // lane value r is T[16 nt + r16][row0 + r]: row-major T
          *reinterpret_cast<bf16x4*>(tout + (16 * nt + r16) * DK + row0) = res;
      }
    }
  }
}

// Element offset of tree level m >= 1 in the tree region (levels 1 .. m-1 before it).
__device__ __host__ inline int64_t tree_level_offset(int64_t BH, int64_t N, int m, int64_t block_size) {
  int64_t off = 0;
  for (int x = 1; x < m; ++x) off += BH * (N >> x) * block_size;
  return off;
}

// ---------------------------------------------------------------------------------------------
// Kernel 3: read-out.  One workgroup (4 waves) per chunk z.  The chunk's Q~ rows are carried
// through its source groups from the lowest set bit of z up: at level j (bit j - 1 set) the rows
// add lambda_t^(log2 C + j) q~_t^T A(G_j) and, if a higher bit follows, become q~^T T(G_j).  The
// node fragments come straight from global memory in the kfrag layout; Q~ lives in LDS (double
// buffered, bf16); wave w owns the output columns DV/4 w .. and the Q~ columns DK/4 w .. .  The
// chunk's intra-chunk output is added at the end and the rows are stored through LDS.
// lambda == NULL: every level weight is 1 (Gated DeltaNet: the whole prefix state).
// ---------------------------------------------------------------------------------------------
template <int C, int DK, int DV, bool HAS_LAMBDA>
__global__ __launch_bounds__(256, 2) void k_gdn_read(const float* __restrict__ lam, const bf* __restrict__ qc_in,
                                                  const bf* __restrict__ pz, const bf* __restrict__ hz,
                                                  const bf* __restrict__ tree, const float* __restrict__ oin_in,
                                                  bf* __restrict__ o, int64_t Tlen, int H, int L, int BH) {
  using MF = Mfma<bf>;
  typedef MF::frag frag;
  constexpr int LOG2C = (C == 16) ? 4 : (C == 32) ? 5 : 6;
  constexpr int KS = DK / 32, RT = C / 16;  // k steps; row tiles (all of them, every wave)
  constexpr int VT = DV / 64, KT = DK / 64; // column tiles of this wave: output, carried Q~
  constexpr int LDQ = DK + 8;
  constexpr int BS = DK * (DK + DV);
  static_assert(C == 64 && VT >= 1 && KT >= 1, "four row tiles, whole column tiles per wave");
  static_assert(2 * C * LDQ * 2 >= C * DV * 4, "the output staging fits the Q~ buffers");
  __shared__ __attribute__((aligned(16))) bf q_s[2][C * LDQ];
  __shared__ float lw_s[HAS_LAMBDA ? C * kMaxJ : 1];

  const int64_t N = Tlen / C;
  const int64_t work = xcd_remap(blockIdx.x, (int64_t)gridDim.x);  // (b h, z): a sequence's chunks on one XCD
  const int64_t z = work % N, bh = work / N;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int64_t cidx = bh * N + z;
  const int64_t tok0 = (int64_t)b * Tlen + z * C;
  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int J = N <= 1 ? 0 : 32 - __builtin_clz((unsigned)(N - 1));

  // node fragments of the level at bit m: A(G) for this wave's output columns, and T(G) for its
  // q~ columns when a higher level follows.  The first level's are loaded before Q~ is staged.
  frag ba[VT][KS], bt[KT][KS];
  auto load_level = [&](int m, bool with_t) {
    const int64_t kblk = (z >> m) - 1;
    const bf *tn, *an;
    if (m == 0) {
      tn = pz + (bh * N + kblk) * (DK * DK);
      an = hz + (bh * N + kblk) * (DK * DV);
    } else {
      tn = tree + tree_level_offset(BH, N, m, BS) + (bh * (N >> m) + kblk) * BS;
      an = tn + DK * DK;
    }
#pragma unroll
    for (int v = 0; v < VT; ++v)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) ba[v][ks] = MF::load(an + (((VT * wave + v) * KS + ks) * 64 + lane) * 8);
    if (with_t) {
#pragma unroll
      for (int v = 0; v < KT; ++v)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) bt[v][ks] = MF::load(tn + (((KT * wave + v) * KS + ks) * 64 + lane) * 8);
    }
  };
  unsigned bits = (unsigned)z;
  if (bits) load_level(__builtin_ctz(bits), (bits & (bits - 1)) != 0);

  for (int x = tid; x < C * DK / 8; x += 256) {
    const int t = x / (DK / 8), c = x % (DK / 8);
    *reinterpret_cast<bf16x8*>(&q_s[0][t * LDQ + 8 * c]) =
        *reinterpret_cast<const bf16x8*>(qc_in + cidx * (C * DK) + t * DK + 8 * c);
  }
  if constexpr (HAS_LAMBDA) {
    for (int x = tid; x < C * J; x += 256) {
      const int t = x / J, jj = x % J;
      lw_s[t * kMaxJ + jj] = lam[((tok0 + t) * H + h) * L + LOG2C + 1 + jj];
    }
  }
  __syncthreads();

  f32x4 acc[RT][VT];
#pragma unroll
  for (int mt = 0; mt < RT; ++mt)
#pragma unroll
    for (int v = 0; v < VT; ++v) acc[mt][v] = f32x4{0.f, 0.f, 0.f, 0.f};
  int cur = 0;
  bool first = true;
  while (bits) {
    const int m = __builtin_ctz(bits);  // tree level of the source group; token level log2 C + m + 1
    bits &= bits - 1;
    if (!first) load_level(m, bits != 0);
    first = false;
    // q~ A(G) for this wave's output columns and, when a higher level follows, q~ T(G) for its
    // q~ columns, from one read of each q~ fragment
    const bf* qs = q_s[cur];
    f32x4 part[RT][VT], qn[RT][KT];
#pragma unroll
    for (int mt = 0; mt < RT; ++mt) {
#pragma unroll
      for (int v = 0; v < VT; ++v) part[mt][v] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int v = 0; v < KT; ++v) qn[mt][v] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int mt = 0; mt < RT; ++mt) {
        const frag a = *reinterpret_cast<const bf16x8*>(&qs[(16 * mt + r16) * LDQ + 32 * ks + 8 * g]);
#pragma unroll
        for (int v = 0; v < VT; ++v) part[mt][v] = MF::mma(a, ba[v][ks], part[mt][v]);
        if (bits) {
#pragma unroll
          for (int v = 0; v < KT; ++v) qn[mt][v] = MF::mma(a, bt[v][ks], qn[mt][v]);
        }
      }
#pragma unroll
    for (int mt = 0; mt < RT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float w = HAS_LAMBDA ? lw_s[(16 * mt + 4 * g + r) * kMaxJ + m] : 1.f;
#pragma unroll
        for (int v = 0; v < VT; ++v) acc[mt][v][r] += w * part[mt][v][r];
      }
    if (bits) {
      bf* qd = q_s[cur ^ 1];
#pragma unroll
      for (int mt = 0; mt < RT; ++mt)
#pragma unroll
        for (int v = 0; v < KT; ++v)
#pragma unroll
          for (int r = 0; r < 4; ++r) qd[(16 * mt + 4 * g + r) * LDQ + 16 * (KT * wave + v) + r16] = static_cast<bf>(qn[mt][v][r]);
      __syncthreads();  // the carried rows complete; every wave is done with the old ones
      cur ^= 1;
    }
  }

  // o = intra-chunk output (stored by the chunk kernel in this accumulator layout) + the levels,
  // rows staged through LDS (over the Q~ buffers)
  const float* oin = oin_in + cidx * (C * DV);
  f32x4 oi[RT][VT];
#pragma unroll
  for (int mt = 0; mt < RT; ++mt)
#pragma unroll
    for (int v = 0; v < VT; ++v)
      oi[mt][v] = *reinterpret_cast<const f32x4*>(oin + ((mt * (DV / 16) + VT * wave + v) * 64 + lane) * 4);
  __syncthreads();
  float* o_s = reinterpret_cast<float*>(&q_s[0][0]);
#pragma unroll
  for (int mt = 0; mt < RT; ++mt)
#pragma unroll
    for (int v = 0; v < VT; ++v)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        o_s[(16 * mt + 4 * g + r) * DV + 16 * (VT * wave + v) + r16] = oi[mt][v][r] + acc[mt][v][r];
  __syncthreads();
  for (int x = tid; x < C * DV / 8; x += 256) {
    const int t = x / (DV / 8), c = 8 * (x % (DV / 8));
    const f32x4 s0 = *reinterpret_cast<const f32x4*>(o_s + t * DV + c);
    const f32x4 s1 = *reinterpret_cast<const f32x4*>(o_s + t * DV + c + 4);
    bf16x8 res;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      res[e] = static_cast<bf>(s0[e]);
      res[4 + e] = static_cast<bf>(s1[e]);
    }
    *reinterpret_cast<bf16x8*>(o + ((tok0 + t) * H + h) * DV + c) = res;
  }
}

}  // namespace gdn

// ---------------------------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------------------------
int64_t gdn_workspace(int64_t B, int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t C, GdnLayout* lay) {
  const int64_t N = T / C, BHN = B * H * N;
  auto al = [](int64_t x) { return (x + 255) & ~int64_t(255); };
  GdnLayout w{};
  int64_t cur = 0;
  w.qc = cur; cur += al(BHN * C * dk * 2);
  w.pz = cur; cur += al(BHN * dk * dk * 2);
  w.hz = cur; cur += al(BHN * dk * dv * 2);
  w.oin = cur; cur += al(BHN * C * dv * 4);
  int64_t blocks = 0;  // tree levels 1 .. J-1 (the source groups of 2 .. 2^(J-1) chunks)
  for (int64_t m = 1; (int64_t(1) << m) < N; ++m) blocks += N >> m;
  w.tree = cur; cur += al(B * H * blocks * dk * (dk + dv) * 2);
  w.total = cur;
  if (lay) *lay = w;
  return cur;
}

// Enqueues the two stages on `st`.  With `ev` non-null, ev[0] is recorded before the chunk
// kernel, ev[1] after it and ev[2] after the tree and read-out kernels (used by the staged entry
// point).
template <int C, int DK, int DV>
hipError_t launch_gdn(const GdnArgs& a, hipStream_t st, hipEvent_t* ev) {
  GdnLayout w;
  gdn_workspace(a.B, a.T, a.H, DK, DV, C, &w);
  char* base = static_cast<char*>(a.workspace);
  __bf16* qc = reinterpret_cast<__bf16*>(base + w.qc);
  __bf16* pz = reinterpret_cast<__bf16*>(base + w.pz);
  __bf16* hz = reinterpret_cast<__bf16*>(base + w.hz);
  float* oin = reinterpret_cast<float*>(base + w.oin);
  const int64_t N = a.T / C;
  const int J = N <= 1 ? 0 : 64 - __builtin_clzll(uint64_t(N - 1));
  // the chunk kernel runs one persistent workgroup per compute unit (its LDS allows no more)
  const int64_t nchunks = a.B * a.H * N;
  int dev = 0, ncu = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || ncu < 1)
    ncu = 256;
  const dim3 g1((unsigned)(nchunks < ncu ? nchunks : ncu));
  const __bf16* q = static_cast<const __bf16*>(a.q);
  const __bf16* k = static_cast<const __bf16*>(a.k);
  const __bf16* v = static_cast<const __bf16*>(a.v);
  __bf16* o = static_cast<__bf16*>(a.o);
  if (ev) (void)hipEventRecord(ev[0], st);
  if (a.lambda)
    hipLaunchKernelGGL((gdn::k_gdn_chunk<C, DK, DV, true>), g1, dim3(64 * gdn::kChunkWaves), 0, st, q, k, v, a.log_alpha, a.beta,
                       a.lambda, qc, pz, hz, oin, a.T, (int)a.H, a.L, nchunks);
  else
    hipLaunchKernelGGL((gdn::k_gdn_chunk<C, DK, DV, false>), g1, dim3(64 * gdn::kChunkWaves), 0, st, q, k, v, a.log_alpha, a.beta,
                       a.lambda, qc, pz, hz, oin, a.T, (int)a.H, a.L, nchunks);
  if (ev) (void)hipEventRecord(ev[1], st);
  // the block tree, one level per launch (level m from level m - 1; level 0 = P_z, H_z)
  __bf16* tree = reinterpret_cast<__bf16*>(base + w.tree);
  const int64_t BH = a.B * a.H, BS = (int64_t)DK * (DK + DV);
  for (int m = 1; m < J; ++m) {
    const __bf16* tin = m == 1 ? pz : tree + gdn::tree_level_offset(BH, N, m - 1, BS);
    const __bf16* ain = m == 1 ? hz : tin + DK * DK;
    const int64_t ts = m == 1 ? DK * DK : BS, as = m == 1 ? DK * DV : BS;
    const int64_t nin = m == 1 ? N : (N >> (m - 1));
    constexpr int split = (DK + DV) / 16 / gdn::kCombineTiles;
    hipLaunchKernelGGL((gdn::k_gdn_combine<DK, DV>), dim3((unsigned)((N >> m) * split), (unsigned)BH), dim3(256), 0, st,
                       tin, ain, ts, as, nin, tree + gdn::tree_level_offset(BH, N, m, BS), N >> m);
  }
  const dim3 g2((unsigned)nchunks);
  if (a.lambda)
    hipLaunchKernelGGL((gdn::k_gdn_read<C, DK, DV, true>), g2, dim3(256), 0, st, a.lambda, qc, pz, hz, tree, oin, o,
                       a.T, (int)a.H, a.L, (int)BH);
  else
    hipLaunchKernelGGL((gdn::k_gdn_read<C, DK, DV, false>), g2, dim3(256), 0, st, a.lambda, qc, pz, hz, tree, oin, o,
                       a.T, (int)a.H, a.L, (int)BH);
  if (ev) (void)hipEventRecord(ev[2], st);
  return hipGetLastError();
}

#define LL_GDN_SHAPES(X) \
  X(64, 64, 64)          \
  X(64, 128, 128)

const GdnEntry* gdn_table(int* n) {
#define LL_ENTRY(C, DK, DV) {C, DK, DV, &launch_gdn<C, DK, DV>},
  static const GdnEntry table[] = {LL_GDN_SHAPES(LL_ENTRY)};
#undef LL_ENTRY
  *n = sizeof(table) / sizeof(table[0]);
  return table;
}

}  // namespace ll
