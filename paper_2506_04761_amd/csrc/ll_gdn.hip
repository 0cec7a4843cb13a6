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
// Kernels: gdn_chunk (one persistent workgroup per compute unit walking its chunks; per chunk the WY
// solve in fp32 by a blocked inversion and all chunk-local products on MFMA, bf16 operands with fp32
// accumulation) and gdn_scan (per (b, h, 16 d_v columns), sequential over the chunks: the level
// states split over the waves by rows and by levels, shared through LDS, P_z / Q~ read once per
// chunk).
#include <type_traits>

#include "ll_device.hpp"
#include "ll_launch.hpp"

namespace ll {

namespace gdn {

constexpr int kMaxJ = 16;      // inter-chunk levels handled by the scan (T <= C * 2^16)
constexpr int kChunkWaves = 8; // waves per gdn_chunk workgroup
constexpr int kSlice = 16;     // d_v columns per scan workgroup
constexpr int kScanWaves = 8;  // waves per scan workgroup
typedef __bf16 bf;

// C = A B over 16x16 output tiles, A [M][K] row-major (lda), Bt = B^T [N][K] row-major (ldb), both
// bf16 in LDS; tiles dealt round-robin to the kChunkWaves waves; epi(mt, nt, acc) consumes each tile
// (lane holds column 16 nt + (lane & 15), rows 16 mt + 4 (lane >> 4) + r).
template <int M, int N, int K, typename Epi>
__device__ inline void gemm_lds(const bf* A, int lda, const bf* Bt, int ldb, Epi epi) {
  using MF = Mfma<bf>;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, r16 = lane & 15, g = lane >> 4;
  constexpr int MT = M / 16, NT = N / 16;
  for (int tile = wave; tile < MT * NT; tile += kChunkWaves) {
    const int mt = tile / NT, nt = tile % NT;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < K / MF::KSTEP; ++ks) {
      const int k0 = ks * MF::KSTEP + g * MF::KPL;
      acc = MF::mma(MF::load(&A[(mt * 16 + r16) * lda + k0]), MF::load(&Bt[(nt * 16 + r16) * ldb + k0]), acc);
    }
    epi(mt, nt, acc);
  }
}

// ---------------------------------------------------------------------------------------------
// Kernel 1: per-chunk WY solve and chunk-local products.  One workgroup (kChunkWaves waves) per chunk.
// Outputs (workspace, per chunk): Qc [C][DK] bf16, P_z [DK][DK] bf16, H_z [DK][DV] bf16,
// intra-chunk output [C][DV] fp32.
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
  __shared__ bf kgt_s[DK * LDC];   // (gamma K)^T
  __shared__ bf kdt_s[DK * LDC];   // (decay-to-end K)^T
  __shared__ bf vt_s[DV * LDC];    // V^T
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
  // memory latency overlaps the current chunk's work.  The 64 lanes of a wave take 64 consecutive
  // tokens of one 8-column piece, so that the transposed (column-major) LDS copies below are
  // written as contiguous runs.
  constexpr int NTH = 64 * kChunkWaves;
  constexpr int NKQ = C * DK / VEC / NTH, NVV = C * DV / VEC / NTH;  // 16-byte pieces per thread
  constexpr int NLW = HAS_LAMBDA ? (C * (LOG2C + 1) + NTH - 1) / NTH : 1;  // lambda values per thread
  static_assert(C * DK / VEC % NTH == 0 && C * DV / VEC % NTH == 0, "whole passes of the workgroup");
  bf16x8 kpre[NKQ], qpre[NKQ], vpre[NVV];
  float la_r = 0.f, bt_r = 0.f, lam_r[NLW];
  auto load_inputs = [&](int64_t it) {
    const int64_t wk = xcd_remap(it, nchunks);
    const int64_t zz = wk % N, bhh = wk / N;
    const int hh = (int)(bhh % H), bb = (int)(bhh / H);
    const int64_t t0 = (int64_t)bb * Tlen + zz * C;
#pragma unroll
    for (int e = 0; e < NKQ; ++e) {
      const int idx = tid + e * NTH, t = idx % C, d0 = (idx / C) * VEC;
      kpre[e] = *reinterpret_cast<const bf16x8*>(k + ((t0 + t) * H + hh) * DK + d0);
      qpre[e] = *reinterpret_cast<const bf16x8*>(q + ((t0 + t) * H + hh) * DK + d0);
    }
#pragma unroll
    for (int e = 0; e < NVV; ++e) {
      const int idx = tid + e * NTH, t = idx % C, d0 = (idx / C) * VEC;
      vpre[e] = *reinterpret_cast<const bf16x8*>(v + ((t0 + t) * H + hh) * DV + d0);
    }
    if (wave == 0 && lane < C) {
      la_r = log_alpha[(t0 + lane) * H + hh] * kLog2e;
      bt_r = beta[(t0 + lane) * H + hh];
    }
    if constexpr (HAS_LAMBDA) {
#pragma unroll
      for (int e = 0; e < NLW; ++e) {
        const int idx = tid + e * NTH, t = idx / (LOG2C + 1), l = idx % (LOG2C + 1);
        if (idx < C * (LOG2C + 1)) lam_r[e] = lam[((t0 + t) * H + hh) * L + l];
      }
    }
  };
  if (blockIdx.x < nchunks) load_inputs(blockIdx.x);
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
    const float la = lane < C ? la_r : 0.f;
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
    const int idx = tid + e * NTH, t = idx % C, d0 = (idx / C) * VEC;
    const bf16x8 kv = kpre[e], qv = qpre[e];
    *reinterpret_cast<bf16x8*>(&k_s[t * LDD + d0]) = kv;
    *reinterpret_cast<bf16x8*>(&q_s[t * LDD + d0]) = qv;
    const float gt = gm_s[t], dt = dc_s[t];
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const float x = static_cast<float>(kv[e]);
      kgt_s[(d0 + e) * LDC + t] = static_cast<bf>(x * gt);
      kdt_s[(d0 + e) * LDC + t] = static_cast<bf>(x * dt);
    }
  }
#pragma unroll
  for (int e = 0; e < NVV; ++e) {
    const int idx = tid + e * NTH, t = idx % C, d0 = (idx / C) * VEC;
    const bf16x8 vv = vpre[e];
#pragma unroll
    for (int e = 0; e < VEC; ++e) vt_s[(d0 + e) * LDC + t] = vv[e];
  }
  if (it + gridDim.x < nchunks) load_inputs(it + gridDim.x);  // the next chunk's, while this one runs
  __syncthreads();
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
  if (wave != 0) {
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
  gemm_lds<C, DK, C>(z_s, LDC, kgt_s, LDC, [&](int mt, int nt, f32x4 acc) {
    bf16x4 w4;
#pragma unroll
    for (int r = 0; r < 4; ++r) w4[r] = static_cast<bf>(acc[r]);
    *reinterpret_cast<bf16x4*>(&wt_s[(nt * 16 + r16) * LDC + mt * 16 + 4 * g]) = w4;
  });
  gemm_lds<C, DV, C>(z_s, LDC, vt_s, LDC, [&](int mt, int nt, f32x4 acc) {
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
  float* oin = oin_out + cidx * (C * DV);
  gemm_lds<C, DV, C>(ph_s, LDC, vt_s, LDC, [&](int mt, int nt, f32x4 acc) {
#pragma unroll
    for (int r = 0; r < 4; ++r) oin[(mt * 16 + 4 * g + r) * DV + nt * 16 + r16] = acc[r];
  });
  bf* qc = qc_out + cidx * (C * DK);
  gemm_lds<C, DK, C>(pg_s, LDC, wt_s, LDC, [&](int mt, int nt, f32x4 acc) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int t = mt * 16 + 4 * g + r, d = nt * 16 + r16;
      const float qv = static_cast<float>(q[((tok0 + t) * H + h) * DK + d]);
      qc[t * DK + d] = static_cast<bf>(gm_s[t] * qv - acc[r]);
    }
  });
  bf* pz = pz_out + cidx * (DK * DK);
  const float gC = gm_s[C - 1];
  gemm_lds<DK, DK, C>(kdt_s, LDC, wt_s, LDC, [&](int mt, int nt, f32x4 acc) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int d = mt * 16 + 4 * g + r, e = nt * 16 + r16;
      pz[d * DK + e] = static_cast<bf>((d == e ? gC : 0.f) - acc[r]);
    }
  });
  bf* hz = hz_out + cidx * (DK * DV);
  gemm_lds<DK, DV, C>(kdt_s, LDC, ut_s, LDC, [&](int mt, int nt, f32x4 acc) {
#pragma unroll
    for (int r = 0; r < 4; ++r) hz[(mt * 16 + 4 * g + r) * DV + nt * 16 + r16] = static_cast<bf>(acc[r]);
  });
  }  // chunk loop
}

// ---------------------------------------------------------------------------------------------
// Kernel 2: level scan.  One workgroup (8 waves) per (b, h, 16 d_v columns), sequential over
// the chunks.  Each level state R_j (d_k x 16) is split over the waves by rows and levels: wave w
// owns rows 32 (w % 4) .. 32 (w % 4) + 31 (DK = 128; 16 rows for DK = 64) of the levels
// j = 1 + (w / 4) + 2 m, in fp32 registers in the MFMA result layout, and reads out chunk row
// tile w % 4 for those levels.  Every wave therefore does the same work.  The propagation
// P_z R_j needs all of R_j's rows as the B operand, so the states of the chunk's start are kept
// in LDS too (bf16, transposed, 16-byte chunks XOR-swizzled by column), rewritten by their owners
// after each step.
// Per step: barrier A (chunk z and the start states are in LDS), propagation and read-out, barrier
// B, then the owners write the new states, P_z and Q~ of chunk z + 1 (loaded into registers during
// the step) go into their single LDS buffers, and the two level groups' partial outputs are added
// to the intra-chunk output.  The H_z and intra-output slices and the level weights come by direct
// global->LDS loads into double buffers, one chunk ahead.
// lambda == NULL: one state (level slot 0 of the first level group), read by every chunk.
// SLOTS: level slots per wave (levels up to 2 SLOTS; 1 for lambda == NULL).
// ---------------------------------------------------------------------------------------------
template <int C, int DK, int DV, bool HAS_LAMBDA, int SLOTS>
__global__ __launch_bounds__(64 * kScanWaves) void k_gdn_scan(const float* __restrict__ lam, const bf* __restrict__ qc_in,
                                                  const bf* __restrict__ pz_in, const bf* __restrict__ hz_in,
                                                  const float* __restrict__ oin_in, bf* __restrict__ o,
                                                  int64_t Tlen, int H, int L, int J) {
  using MF = Mfma<bf>;
  constexpr int LOG2C = (C == 16) ? 4 : (C == 32) ? 5 : 6;
  constexpr int MTD = DK / 16;          // 16-row tiles of a state
  constexpr int MPW = MTD / 4;          // of them owned by a wave
  constexpr int KS = DK / 32;           // k steps over d_k
  constexpr int NSL = DV / kSlice;
  constexpr int LPW = SLOTS;                       // level slots per wave
  static_assert(HAS_LAMBDA ? 2 * SLOTS <= kMaxJ : SLOTS == 1, "level slots");
  constexpr int NLV = HAS_LAMBDA ? kMaxJ : 1;      // level states kept in LDS
  constexpr int NT = 64 * kScanWaves;
  constexpr int CPR = DK / 8;           // 16-byte chunks per state column / per P_z or Q~ row
  constexpr int PZC = DK * CPR / NT, QCC = C * CPR / NT;  // chunks per thread of P_z, Q~
  static_assert(kSlice == 16 && kScanWaves == 8 && C == 64, "4 row groups x 2 level groups, 4 chunk row tiles");
  static_assert(MTD % 4 == 0 && PZC >= 1 && QCC >= 1 && DK * CPR % NT == 0 && C * CPR % NT == 0, "tile split");
  __shared__ bf pz_s[DK * DK];                       // swizzled rows
  __shared__ bf qc_s[C * DK];                        // swizzled rows
  __shared__ bf rs_s[NLV * kSlice * DK];             // [level][column][row], swizzled chunks
  __shared__ bf hz_s[2][DK * kSlice];                // [row][16]
  __shared__ float oin_s[2][C * kSlice];             // [t][16]
  __shared__ float lw_s[2][HAS_LAMBDA ? C * kMaxJ : 1];
  __shared__ float part_s[2 * C * kSlice];           // [level group][t][16]

  const int64_t N = Tlen / C;
  const int64_t work = xcd_remap(blockIdx.x, (int64_t)gridDim.x);  // (b, h, slice)
  const int sl = (int)(work % NSL);
  const int64_t bh = work / NSL;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rg = wave & 3, lgp = wave >> 2;  // row group, level group
  const int p0 = sl * kSlice;

  // state entry (level slot l, column c, row) in rs_s
  auto rs_off = [](int l, int c, int row) {
    return (l * kSlice + c) * DK + ((((row >> 3) ^ c) & (CPR - 1)) << 3) + (row & 7);
  };
  // the small per-chunk inputs into buffer half `buf`
  auto fetch = [&](int64_t z, int buf) {
    const int64_t cidx = bh * N + z;
    const int64_t tok0 = (int64_t)b * Tlen + z * C;
    const bf* hs = hz_in + cidx * (DK * DV) + p0;
    lds_gather16<NT>(hz_s[buf], DK * 2, [&](int q) { return hs + (q >> 1) * DV + (q & 1) * 8; });
    const float* os = oin_in + cidx * (C * DV) + p0;
    lds_gather16<NT>(oin_s[buf], C * 4, [&](int q) { return os + (q >> 2) * DV + (q & 3) * 4; });
    if constexpr (HAS_LAMBDA) {
      if (J > 0) {  // weights of levels LOG2C + 1 .. LOG2C + J (slots jj >= J repeat level J)
        const float* ls = lam + (tok0 * H + h) * L + LOG2C + 1;
        lds_gather4<NT>(lw_s[buf], C * kMaxJ, [&](int q) {
          const int t = q / kMaxJ, jj = q % kMaxJ;
          return ls + (int64_t)t * H * L + (jj < J ? jj : J - 1);
        });
      }
    }
  };
  // P_z and Q~ of chunk z into registers, then (once the step's readers are done) into LDS
  bf16x8 pzr[PZC], qcr[QCC];
  auto load_big = [&](int64_t z) {
    const int64_t cidx = bh * N + z;
#pragma unroll
    for (int e = 0; e < PZC; ++e) {
      const int x = e * NT + tid;
      pzr[e] = *reinterpret_cast<const bf16x8*>(pz_in + cidx * (DK * DK) + (x / CPR) * DK + (x % CPR) * 8);
    }
#pragma unroll
    for (int e = 0; e < QCC; ++e) {
      const int x = e * NT + tid;
      qcr[e] = *reinterpret_cast<const bf16x8*>(qc_in + cidx * (C * DK) + (x / CPR) * DK + (x % CPR) * 8);
    }
  };
  auto store_big = [&]() {
#pragma unroll
    for (int e = 0; e < PZC; ++e) {
      const int x = e * NT + tid;
      *reinterpret_cast<bf16x8*>(pz_s + swz<DK>(x / CPR, x % CPR)) = pzr[e];
    }
#pragma unroll
    for (int e = 0; e < QCC; ++e) {
      const int x = e * NT + tid;
      *reinterpret_cast<bf16x8*>(qc_s + swz<DK>(x / CPR, x % CPR)) = qcr[e];
    }
  };

  f32x4 R[LPW][MPW];
#pragma unroll
  for (int m = 0; m < LPW; ++m)
#pragma unroll
    for (int i = 0; i < MPW; ++i) R[m][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int x = tid; x < NLV * kSlice * DK / 8; x += NT) reinterpret_cast<bf16x8*>(rs_s)[x] = bf16x8{};
  load_big(0);
  store_big();
  fetch(0, 0);
  for (int64_t z = 0; z < N; ++z) {
    const int buf = (int)(z & 1);
    const int64_t tok0 = (int64_t)b * Tlen + z * C;
    wait_vmem();
    __syncthreads();  // A: chunk z and the start states in LDS; every wave is done with the other half
    if (z + 1 < N) {
      fetch(z + 1, buf ^ 1);
      load_big(z + 1);
    }

    f32x4 out = {0.f, 0.f, 0.f, 0.f};  // chunk rows 16 rg + 4g + r, column p0 + r16
    // this lane's entries of H_z (rows 16 (MPW rg + i) + 4g + r, column p0 + r16)
    f32x4 hzv[MPW];
#pragma unroll
    for (int i = 0; i < MPW; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        hzv[i][r] = static_cast<float>(hz_s[buf][(16 * (MPW * rg + i) + 4 * g + r) * kSlice + r16]);

#pragma unroll
    for (int m = 0; m < LPW; ++m) {
      int j;
      bool reader, source, restart;
      if constexpr (HAS_LAMBDA) {
        j = 1 + lgp + 2 * m;
        if (j > J) continue;
        reader = (z >> (j - 1)) & 1;
        source = !reader;
        restart = (z & ((int64_t(1) << j) - 1)) == 0;
      } else {
        if (lgp != 0) continue;
        j = 0;
        reader = z > 0;
        source = true;
        restart = z == 0;
      }
      const int slot = HAS_LAMBDA ? j - 1 : 0;
      // B fragments of R_j at the chunk's start: column r16, rows 32 ks + 8 g .. + 7
      bf16x8 rb[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        rb[ks] = *reinterpret_cast<const bf16x8*>(rs_s + rs_off(slot, r16, 32 * ks + 8 * g));
      if (reader) {
        f32x4 tmp = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) tmp = MF::mma(frag_along_row_swz<DK>(qc_s, 16 * rg, 4 * ks), rb[ks], tmp);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = 16 * rg + 4 * g + r;
          const float wgt = HAS_LAMBDA ? lw_s[buf][t * kMaxJ + (j - 1)] : 1.f;
          out[r] += wgt * tmp[r];
        }
      }
#pragma unroll
      for (int i = 0; i < MPW; ++i) {
        if (restart) {
          R[m][i] = hzv[i];
        } else {
          f32x4 acc = source ? hzv[i] : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            acc = MF::mma(frag_along_row_swz<DK>(pz_s, 16 * (MPW * rg + i), 4 * ks), rb[ks], acc);
          R[m][i] = acc;
        }
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) part_s[(lgp * C + 16 * rg + 4 * g + r) * kSlice + r16] = out[r];
    __syncthreads();  // B: every read of the start states, P_z and Q~ is done; partial outputs complete

    // the new states (rows 16 (MPW rg + i) + 4g .. + 3 of column r16: 8 bytes each)
#pragma unroll
    for (int m = 0; m < LPW; ++m) {
      const int j = HAS_LAMBDA ? 1 + lgp + 2 * m : 0;
      if (HAS_LAMBDA ? j > J : lgp != 0) continue;
      const int slot = HAS_LAMBDA ? j - 1 : 0;
#pragma unroll
      for (int i = 0; i < MPW; ++i) {
        bf16x4 v4;
#pragma unroll
        for (int r = 0; r < 4; ++r) v4[r] = static_cast<bf>(R[m][i][r]);
        *reinterpret_cast<bf16x4*>(rs_s + rs_off(slot, r16, 16 * (MPW * rg + i) + 4 * g)) = v4;
      }
    }
    if (z + 1 < N) store_big();
    for (int idx = tid; idx < C * kSlice; idx += NT) {
      const int t = idx / kSlice, p = idx % kSlice;
      float acc = oin_s[buf][idx] + part_s[idx];
      if constexpr (HAS_LAMBDA) acc += part_s[C * kSlice + idx];
      o[((tok0 + t) * H + h) * DV + p0 + p] = static_cast<bf>(acc);
    }
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
  w.total = cur;
  if (lay) *lay = w;
  return cur;
}

// Enqueues the two stages on `st`.  With `ev` non-null, ev[0] is recorded before the chunk
// kernel, ev[1] between the kernels and ev[2] after the scan (used by the staged entry point).
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
  const dim3 g1((unsigned)(nchunks < ncu ? nchunks : ncu)), g2((unsigned)(a.B * a.H * (DV / gdn::kSlice)));
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
  if (a.lambda && J <= 8)
    hipLaunchKernelGGL((gdn::k_gdn_scan<C, DK, DV, true, 4>), g2, dim3(64 * gdn::kScanWaves), 0, st, a.lambda, qc, pz,
                       hz, oin, o, a.T, (int)a.H, a.L, J);
  else if (a.lambda)
    hipLaunchKernelGGL((gdn::k_gdn_scan<C, DK, DV, true, gdn::kMaxJ / 2>), g2, dim3(64 * gdn::kScanWaves), 0, st,
                       a.lambda, qc, pz, hz, oin, o, a.T, (int)a.H, a.L, J);
  else
    hipLaunchKernelGGL((gdn::k_gdn_scan<C, DK, DV, false, 1>), g2, dim3(64 * gdn::kScanWaves), 0, st, a.lambda, qc, pz,
                       hz, oin, o, a.T, (int)a.H, a.L, J);
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
