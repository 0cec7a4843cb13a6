// Log-linear Mamba-2 backward: the gradients of O = (Q K^T (.) M^S (.) M^H) V (Sec. 3.4) with
// respect to q, k, v, the log-gates and lambda, computed chunkwise in the forward's tiles of R
// rows (Sec. 3.3 organisation; the gradient formulas follow from the forward by the chain rule).
//
// Per (b, h), with w(t, s) = lambda_t^(l(t, s)) exp(cum_t - cum_s) for s <= t, P = Q K^T and
// G = dO V^T:
//   dQ = (w (.) G) K,   dK = (w (.) G)^T Q,   dV = (w (.) P)^T dO,
//   dlambda_t^(l) = sum over s at level l of exp(cum_t - cum_s) P[t, s] G[t, s],
//   dlog_alpha_tau = sum_{t >= tau} (q_t . dq_t - k_t . dk_t).
//
// Query side (dq, dlambda): pairs inside a tile densely; pairs in different tiles through the
// forward's level summaries U_j (d_v x d_k), which tile u reads at every set bit j-1 of u:
//   dq_t += lambda_t^(log2 R + j) exp2(cl_t + gap_j) U_j^T dO_t,
//   dlambda_t^(log2 R + j) = exp2(cl_t + gap_j) dO_t . (U_j q_t).
// Key side (dk, dv): the same pairs seen from the key.  lambda belongs to the later (query)
// token, so every level needs summaries of its own: key tile s with bit j-1 clear sends its keys
// to the group G'_j(s) of the 2^(j-1) tiles that follow s's aligned 2^(j-1)-tile block, and
//   D_j = sum_{t in G'_j} lambda_t^(log2 R + j) exp2(c_t) dO_t q_t^T   (d_v x d_k; c_t = summed
//         log2-gates from the start of G'_j through t),
//   dk_s += exp2(tot_s - cl_s + gap'_j) D_j^T v_s,   dv_s += exp2(...) D_j k_s,
// gap'_j being the summed gates of the tiles strictly between s and G'_j: the groups of s's
// lower key-side levels.  One D_j serves both dk and dv.
//
// Kernels, in stream order:
//   (forward block_state and level scan)  the summaries U_j and the tile gates
//   k_rev_state   one workgroup per (level, up to 8 tiles of one group): D_j of the groups of at
//                 most 8 tiles, fp32 partial sums over 8-tile regions of the larger groups
//   k_rev_reduce  the groups of >= 16 tiles: sums of their regions' partials
//   k_bwd_dq      per tile: dq, dlambda and q . dq
//   k_bwd_dkv     per tile: dk, dv, and the tile-local suffix sums of q . dq - k . dk into dlog_alpha
//   k_bwd_dgate   adds the sums of all later tiles to dlog_alpha
#include <type_traits>

#include "ll_mamba2_common.hpp"

namespace ll {

namespace {

constexpr int kRegionTiles = 8;   // tiles per region (the unit of k_rev_state's partial sums)
constexpr int kRevThreads = 512;  // k_rev_state workgroup: 8 waves

template <int R>
struct Log2 {
  static constexpr int v = R == 64 ? 6 : R == 128 ? 7 : -1;
};

// Device view of the key-side level summaries.  Level j's groups are the upper halves of the
// aligned 2^j-tile blocks whose first tile exists; group m starts at tile (2m + 1) 2^(j-1).
template <typename T>
struct RevNodes {
  T* d;          // [BH][nd] D_j per group, [p][n] = d_v x d_k, storage type
  float* dtot;   // [BH][nd] summed log2-gates of each group
  float* part;   // [BH][npart] fp32 sums over one 8-tile region of a level >= 5 group, [p][n]
  int64_t N, NR, nd, npart;
  __device__ __host__ static int64_t groups(int64_t N, int j) {
    const int64_t a = (N - 1) >> (j - 1);
    return a >= 1 ? (a + 1) / 2 : 0;
  }
  __device__ __host__ int64_t slot(int64_t bh, int j, int64_t m) const {
    int64_t off = 0;
    for (int l = 1; l < j; ++l) off += groups(N, l);
    return bh * nd + off + m;
  }
  // regions rg < NR with bit j - 4 set: the regions of level-j groups (j >= 5)
  __device__ __host__ static int64_t parts(int64_t NR, int j) {
    const int64_t lo = int64_t(1) << (j - 4), rem = NR & (2 * lo - 1);
    return ((NR >> (j - 3)) << (j - 4)) + (rem > lo ? rem - lo : 0);
  }
  __device__ __host__ int64_t pslot(int64_t bh, int j, int64_t rg) const {
    int64_t off = 0;
    for (int l = 5; l < j; ++l) off += parts(NR, l);
    const int64_t lo = int64_t(1) << (j - 4);
    return bh * npart + off + ((rg >> (j - 3)) << (j - 4)) + (rg & (lo - 1));
  }
};

// Whether key tile s sends its keys to a level-j group (bit j-1 clear, and the group exists).
__device__ inline bool key_level(int64_t s, int j, int64_t N) {
  return !((s >> (j - 1)) & 1) && ((((s >> (j - 1)) | 1) << (j - 1)) < N);
}

// Sum of a value over the 4 lane groups (g = lane / 16) holding the rows of one MFMA column.
__device__ inline float sum_over_groups(float x) {
  x += __shfl_xor(x, 16, 64);
  x += __shfl_xor(x, 32, 64);
  return x;
}

// Adds x to acc[lv] for a level lv < NL known only at run time.
template <int NL>
__device__ inline void add_level(float (&acc)[NL], int lv, float x) {
#pragma unroll
  for (int l = 0; l < NL; ++l)
    if (l == lv) acc[l] += x;
}

// Operand fragment with its k slots running down rows r0 .. r0 + KSTEP - 1 of a row-major
// matrix in LDS (column col0 + lane % 16).  The k slots are assigned the way a B operand built
// from MFMA result tiles assigns them (bf16: two 16-row result tiles per k step, fp32: one k step
// per result row r of a 16-row tile), so such pairs contract correctly.
template <typename T>
__device__ inline typename Mfma<T>::frag frag_rows(const T* m, int ld, int r0, int col0, int r);
template <>
__device__ inline bf16x8 frag_rows<__bf16>(const __bf16* m, int ld, int r0, int col0, int) {
  return frag_down_rows(m, ld, r0, col0);
}
template <>
__device__ inline float frag_rows<float>(const float* m, int ld, int r0, int col0, int r) {
  const int lane = threadIdx.x & 63;
  return m[(r0 + 4 * (lane >> 4) + r) * ld + col0 + (lane & 15)];
}

// B operand from result-layout values: bf16 packs two 16-row tiles (slots 0-3 from a, 4-7 from
// b); fp32 takes value r of one tile.
__device__ inline bf16x8 pack_rl(const f32x4& a, const f32x4& b) {
  bf16x8 f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    f[r] = static_cast<__bf16>(a[r]);
    f[4 + r] = static_cast<__bf16>(b[r]);
  }
  return f;
}

// Copies rows 0 .. R-1 of a [rows, H, D] tensor (tile rows from row0; rows at or beyond nrow
// repeat row nrow - 1) into a row-major LDS tile of row stride LD.
template <typename T, int D, int LD, int R, int NT>
__device__ inline void load_tile(T* dst, const T* __restrict__ src, int64_t row0, int nrow, int H, int h) {
  typedef typename Vec16<T>::type V16;
  constexpr int VEC = Vec16<T>::N, PER = D / VEC;
  for (int idx = threadIdx.x; idx < R * PER; idx += NT) {
    const int r = idx / PER, c = idx % PER;
    const int rs = r < nrow ? r : nrow - 1;
    *reinterpret_cast<V16*>(&dst[r * LD + c * VEC]) =
        *reinterpret_cast<const V16*>(src + ((row0 + rs) * H + h) * D + c * VEC);
  }
}

// lambda of the tile's rows into dst[r * L + l] (rows < nrow).
template <int NT>
__device__ inline void load_lambda(float* dst, const float* __restrict__ lam, int64_t row0, int nrow, int H, int h,
                                   int L) {
  for (int idx = threadIdx.x; idx < nrow * L; idx += NT) {
    const int r = idx / L, l = idx % L;
    dst[idx] = lam[((row0 + r) * H + h) * L + l];
  }
}

}  // namespace

// ---------------------------------------------------------------------------------------------
// k_rev_state: one workgroup per (b, h, 8-tile region rg, item), one tile per step.  Items 0-3: level 1, tile
// 8 rg + 2 i + 1; items 4-5: level 2, tiles 8 rg + 4 (i - 4) + {2, 3}; item 6: level 3, tiles
// 8 rg + 4 .. 8 rg + 7; item 3 + j (j >= 4): level j, the whole region, present when bit j - 4 of
// rg is set.  Each item forms sum_t w_t dO_t q_t^T over its tiles with
// w_t = lambda_t^(log2 R + j) exp2(c_t), c_t the summed log2-gates from the item's first row through
// t, one tile per step: (w q) and dO staged in LDS, both MFMA operands read down the token rows.
// Items of levels <= 4 cover their whole group and write D_j; the others write fp32 partials.
// ---------------------------------------------------------------------------------------------
template <typename T, int C, int DK, int DV>
__global__ __launch_bounds__(kRevThreads) void k_rev_state(const T* __restrict__ q, const T* __restrict__ dout,
                                                           const float* __restrict__ lam, Nodes<T> nodes,
                                                           RevNodes<T> rev, int64_t Tlen, int H, int Hqk, int L,
                                                           int J, int items) {
  using M = Mfma<T>;
  typedef typename Vec16<T>::type V16;
  constexpr int R = tile_rows(C), LOG2R = Log2<R>::v;
  constexpr int VEC = Vec16<T>::N;
  constexpr int LDQ = DK + 16, LDO = DV + 16;
  constexpr int MT = DV / 16, NTN = DK / 16;
  constexpr int NW = kRevThreads / 64;
  constexpr int WM = MT >= 2 ? 2 : 1;
  constexpr int WN = (NW / WM) < NTN ? (NW / WM) : NTN;
  constexpr int TM = MT / WM, TN = NTN / WN;
  constexpr int SZ = DK * DV;
  constexpr int HALVES = R / kKB;  // 64-row register blocks per tile (one tile per step)
  static_assert(SZ <= R * LDQ, "the finished summary is staged in the Q buffer");
  __shared__ T q_s[R * LDQ];
  __shared__ T o_s[R * LDO];
  __shared__ float w_s[R];
  T* out_s = q_s;

  const int64_t N = rev.N, NR = rev.NR;
  const int64_t work = xcd_remap(blockIdx.x, (int64_t)gridDim.x);  // logical order (b, h, rg, item)
  const int it = (int)(work % items);
  const int64_t rg = (work / items) % NR;
  const int64_t bh = work / (items * NR);
  const int h = (int)(bh % H), b = (int)(bh / H);
  int j, nt;
  int64_t u0;
  if (it < 4) { j = 1; u0 = kRegionTiles * rg + 2 * it + 1; nt = 1; }
  else if (it < 6) { j = 2; u0 = kRegionTiles * rg + 4 * (it - 4) + 2; nt = 2; }
  else if (it == 6) { j = 3; u0 = kRegionTiles * rg + 4; nt = 4; }
  else { j = it - 3; u0 = kRegionTiles * rg; nt = kRegionTiles; }
  if (j > J || u0 >= N) return;
  if (j >= 4 && !((rg >> (j - 4)) & 1)) return;
  if (u0 + nt > N) nt = (int)(N - u0);
  const int hq = h / (H / Hqk);  // this head's query/key head

  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool active = wave < WM * WN;
  const int wm = wave / WN, wn = wave % WN;
  const int nsteps = nt;
  auto nrow_of = [&](int64_t u) { return (int)((Tlen - u * R) < R ? (Tlen - u * R) : R); };
  auto tile_row0 = [&](int64_t u) { return (int64_t)b * Tlen + u * R; };

  RowBlock<T, DK, kRevThreads> qr[HALVES];
  RowBlock<T, DV, kRevThreads> dr[HALVES];
  float wv = 0.f;
  float base = 0.f;  // summed log2-gates of the item's tiles before the current one
  // loads of step s = tile u0 + s (rows past the sequence get weight 0)
  auto load_step = [&](int s) {
    const int64_t u = u0 + s;
#pragma unroll
    for (int x = 0; x < HALVES; ++x) {
      qr[x].load(q, tile_row0(u), x * kKB, nrow_of(u), Hqk, hq);
      dr[x].load(dout, tile_row0(u), x * kKB, nrow_of(u), H, h);
    }
    if (tid < R) {
      const float c = base + nodes.cl[(bh * N + u) * R + tid];
      wv = tid < nrow_of(u) ? lam[((tile_row0(u) + tid) * H + h) * L + LOG2R + j] * fast_exp2(c) : 0.f;
    }
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int jn = 0; jn < TN; ++jn) acc[i][jn] = f32x4{0.f, 0.f, 0.f, 0.f};

  load_step(0);
  for (int s = 0; s < nsteps; ++s) {
    __syncthreads();  // previous step's readers are done
    if (tid < R) w_s[tid] = wv;
#pragma unroll
    for (int x = 0; x < HALVES; ++x) dr[x].store_rows(o_s + x * kKB * LDO, LDO);
    __syncthreads();
#pragma unroll
    for (int x = 0; x < HALVES; ++x) qr[x].store_rows_scaled(q_s + x * kKB * LDQ, LDQ, w_s + x * kKB);
    base += nodes.t1[bh * N + u0 + s];
    if (s + 1 < nsteps) load_step(s + 1);
    __syncthreads();
    if (active) {
#pragma unroll
      for (int ks = 0; ks < R / M::KSTEP; ++ks) {
        typename M::frag bf[TN];
#pragma unroll
        for (int jn = 0; jn < TN; ++jn) {
          const int n0 = (wn * TN + jn) * 16;
          if constexpr (M::KPL == 8) bf[jn] = frag_down_rows(q_s, LDQ, ks * 32, n0);
          else bf[jn] = q_s[(ks * 4 + g) * LDQ + n0 + r16];
        }
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int p0 = (wm * TM + i) * 16;
          typename M::frag af;
          if constexpr (M::KPL == 8) af = frag_down_rows(o_s, LDO, ks * 32, p0);
          else af = o_s[(ks * 4 + g) * LDO + p0 + r16];
#pragma unroll
          for (int jn = 0; jn < TN; ++jn) acc[i][jn] = M::mma(af, bf[jn], acc[i][jn]);
        }
      }
    }
  }

  if (j <= 4) {
    const int64_t sl = rev.slot(bh, j, u0 >> j);
    __syncthreads();  // every wave is done with the Q buffer
    if (active) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int jn = 0; jn < TN; ++jn)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int p = (wm * TM + i) * 16 + 4 * g + r, n = (wn * TN + jn) * 16 + r16;
            out_s[p * DK + n] = from_f32<T>(acc[i][jn][r]);
          }
    }
    __syncthreads();
    T* dst = rev.d + sl * SZ;
    for (int idx = tid; idx < SZ / VEC; idx += kRevThreads)
      *reinterpret_cast<V16*>(dst + idx * VEC) = *reinterpret_cast<const V16*>(&out_s[idx * VEC]);
    if (tid == 0) rev.dtot[sl] = base;
  } else if (active) {
    float* dst = rev.part + rev.pslot(bh, j, rg) * SZ;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int jn = 0; jn < TN; ++jn)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int p = (wm * TM + i) * 16 + 4 * g + r, n = (wn * TN + jn) * 16 + r16;
          dst[p * DK + n] = acc[i][jn][r];
        }
  }
}

// ---------------------------------------------------------------------------------------------
// k_rev_reduce: grid (SZ / 1024 entry blocks, level >= 5 groups, B * H); each thread sums four
// entries of one group's region partials, region by region, each weighted by the gates of the
// group's regions before it.
// ---------------------------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_rev_reduce(Nodes<T> nodes, RevNodes<T> rev, int J, int SZ) {
  const int64_t N = rev.N, NR = rev.NR;
  const int64_t bh = blockIdx.z;
  int64_t y = blockIdx.y;
  int j = 5;
  for (; j <= J; ++j) {
    const int64_t ng = RevNodes<T>::groups(N, j);
    if (y < ng) break;
    y -= ng;
  }
  if (j > J) return;
  const int64_t first = (2 * y + 1) << (j - 1);
  const int64_t rg0 = first / kRegionTiles;
  int64_t nreg = int64_t(1) << (j - 4);
  if (rg0 + nreg > NR) nreg = NR - rg0;
  const int e0 = (blockIdx.x * 256 + threadIdx.x) * 4;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float base = 0.f;
  // four regions per step: their partials are loaded together, then added in region order
  constexpr int U = 4;
  for (int64_t r = 0; r < nreg; r += U) {
    f32x4 xs[U];
    float wq[U];
#pragma unroll
    for (int q = 0; q < U; ++q) {
      const int64_t rgn = rg0 + r + q;
      const bool live = r + q < nreg;
      xs[q] = live && e0 < SZ ? *reinterpret_cast<const f32x4*>(rev.part + rev.pslot(bh, j, rgn) * SZ + e0)
                              : f32x4{0.f, 0.f, 0.f, 0.f};
      wq[q] = fast_exp2(base);
      if (live) {
        const int64_t x1 = (rgn + 1) * kRegionTiles < N ? (rgn + 1) * kRegionTiles : N;
        for (int64_t x = rgn * kRegionTiles; x < x1; ++x) base += nodes.t1[bh * N + x];
      }
    }
#pragma unroll
    for (int q = 0; q < U; ++q)
      if (r + q < nreg) acc += wq[q] * xs[q];
  }
  const int64_t sl = rev.slot(bh, j, y);
  if (e0 < SZ)
#pragma unroll
    for (int e = 0; e < 4; ++e) rev.d[sl * SZ + e0 + e] = from_f32<T>(acc[e]);
  if (blockIdx.x == 0 && threadIdx.x == 0) rev.dtot[sl] = base;
}

// ---------------------------------------------------------------------------------------------
// k_bwd_dq: one workgroup of R/16 waves per (b, h, tile); wave w owns query rows 16 w .. 16 w + 15,
// one per MFMA column (lane % 16).  K and V of the tile resident in LDS.
//   intra: S^T = K Q^T and G^T = V dO^T per 16-key tile; weights lambda_i^(l) exp2(cl_i - cl_j);
//          dq^T += K^T (w (.) G)^T; dlambda_i^(l) += exp2(cl_i - cl_j) S G, summed per level;
//   inter: per level read, U_j copied into LDS: y^T = U_j Q^T (dlambda = dO . y), and
//          dq^T += (lambda exp2(cl + gap)) U_j^T dO^T.
// ---------------------------------------------------------------------------------------------
template <typename T, int C, int DK, int DV>
__global__ __launch_bounds__(4 * tile_rows(C)) void k_bwd_dq(const T* __restrict__ q, const T* __restrict__ k,
                                                            const T* __restrict__ v, const T* __restrict__ dout,
                                                            const float* __restrict__ log_alpha,
                                                            const float* __restrict__ lam, Nodes<T> nodes,
                                                            T* __restrict__ dq, float* __restrict__ dlam,
                                                            float* __restrict__ qdq, int64_t Tlen, int H, int Hqk, int L,
                                                            int J) {
  using M = Mfma<T>;
  typedef typename Vec16<T>::type V16;
  constexpr int R = tile_rows(C), LOG2R = Log2<R>::v, NW = R / 16, NT = 64 * NW;
  constexpr int VEC = Vec16<T>::N;
  constexpr int LDK = DK + 16, LDV = DV + 16;
  constexpr int KSK = DK / M::KSTEP, KSV = DV / M::KSTEP, MTK = DK / 16, MTV = DV / 16;
  constexpr int SZ = DK * DV;
  constexpr int NL = LOG2R + 1;  // levels inside a tile
  static_assert(DV <= R, "a summary fits in the K region");
  __shared__ T k_s[R * LDK];
  __shared__ T v_s[R * LDV];
  __shared__ float cl_s[R];
  __shared__ float wsum_s[4];
  __shared__ float lam_s[R * kMaxLevels];
  __shared__ float dl_s[R * kMaxLevels];
  T* u_s = k_s;

  const int64_t N = (Tlen + R - 1) / R;
  const int64_t work = xcd_remap(blockIdx.x, (int64_t)gridDim.x);  // logical order (b, h, u)
  const int u = (int)(work % N);
  const int64_t bh = work / N;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t row0 = (int64_t)b * Tlen + (int64_t)u * R;
  const int nrow = (int)((Tlen - (int64_t)u * R) < R ? (Tlen - (int64_t)u * R) : R);
  const int i = 16 * wave + r16;  // this lane's query row
  const bool rowok = i < nrow;
  const int64_t qrow = (row0 + (rowok ? i : 0)) * H + h;
  const int hq = h / (H / Hqk);  // this head's query/key head
  const int64_t qkrow = (row0 + (rowok ? i : 0)) * Hqk + hq;

  const float la = tile_gate<R>(log_alpha, row0, nrow, H, h);
  load_tile<T, DK, LDK, R, NT>(k_s, k, row0, nrow, Hqk, hq);
  load_tile<T, DV, LDV, R, NT>(v_s, v, row0, nrow, H, h);
  load_lambda<NT>(lam_s, lam, row0, nrow, H, h, L);
  for (int x = tid; x < R * kMaxLevels; x += NT) dl_s[x] = 0.f;

  typename M::frag qf[KSK], df[KSV];
#pragma unroll
  for (int ks = 0; ks < KSK; ++ks)
    qf[ks] = rowok ? M::load(q + qkrow * DK + ks * M::KSTEP + g * M::KPL) : typename M::frag{};
#pragma unroll
  for (int ks = 0; ks < KSV; ++ks)
    df[ks] = rowok ? M::load(dout + qrow * DV + ks * M::KSTEP + g * M::KPL) : typename M::frag{};
  f32x4 dorl[MTV];  // dO of row i at d_v entries 16 mt + 4 g + r
#pragma unroll
  for (int mt = 0; mt < MTV; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) dorl[mt][r] = rowok ? to_f32(dout[qrow * DV + 16 * mt + 4 * g + r]) : 0.f;

  tile_cumsum_of<R>(la, nrow, cl_s, wsum_s);  // barriers: the LDS tiles are visible after it
  const float cli = cl_s[i];
  const float* lrow = &lam_s[(rowok ? i : 0) * L];

  f32x4 acc[MTK];
#pragma unroll
  for (int mt = 0; mt < MTK; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  float dl[NL];
#pragma unroll
  for (int l = 0; l < NL; ++l) dl[l] = 0.f;

  // weights of one 16-key tile KT <= wave, in the result layout (key 16 KT + 4 g + r, query i)
  auto key_tile = [&](int KT, f32x4& wg) {
    f32x4 s = {0.f, 0.f, 0.f, 0.f}, gg = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KSK; ++ks)
      s = M::mma(M::load(&k_s[(KT * 16 + r16) * LDK + ks * M::KSTEP + g * M::KPL]), qf[ks], s);
#pragma unroll
    for (int ks = 0; ks < KSV; ++ks)
      gg = M::mma(M::load(&v_s[(KT * 16 + r16) * LDV + ks * M::KSTEP + g * M::KPL]), df[ks], gg);
    if (KT < wave) {
      const int lv = level_local(16 * wave, 16 * KT);  // one level for the whole 16 x 16 tile
      const float lw = rowok ? lrow[lv] : 0.f;
      float pg = 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float e = fast_exp2(cli - cl_s[16 * KT + 4 * g + r]);
        pg += e * s[r] * gg[r];
        wg[r] = lw * e * gg[r];
      }
      add_level(dl, lv, pg);
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int jj = 16 * KT + 4 * g + r;
        const bool ok = jj <= i && rowok;
        const int lv = level_local(i, jj);
        const float e = ok ? fast_exp2(cli - cl_s[jj]) : 0.f;
        add_level(dl, ok ? lv : 0, e * s[r] * gg[r]);
        wg[r] = ok ? lrow[lv] * e * gg[r] : 0.f;
      }
    }
  };

  if constexpr (M::KPL == 8) {
    for (int st = 0; 2 * st <= wave; ++st) {
      f32x4 w0, w1 = {0.f, 0.f, 0.f, 0.f};
      key_tile(2 * st, w0);
      if (2 * st + 1 <= wave) key_tile(2 * st + 1, w1);
      const bf16x8 bp = pack_rl(w0, w1);
#pragma unroll
      for (int mt = 0; mt < MTK; ++mt) acc[mt] = M::mma(frag_rows<T>(k_s, LDK, 32 * st, 16 * mt, 0), bp, acc[mt]);
    }
  } else {
    for (int KT = 0; KT <= wave; ++KT) {
      f32x4 w0;
      key_tile(KT, w0);
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int mt = 0; mt < MTK; ++mt)
          acc[mt] = M::mma(frag_rows<T>(k_s, LDK, 16 * KT, 16 * mt, r), w0[r], acc[mt]);
    }
  }
#pragma unroll
  for (int l = 0; l < NL; ++l) {
    const float x = sum_over_groups(dl[l]);
    if (g == 0 && rowok && l < L) dl_s[i * L + l] = x;
  }

  // ---- inter-tile levels (set bits of u) through the forward's summaries
  const float gapv = level_gaps(nodes, bh, N, u, J);
  for (int j = 1; j <= J; ++j) {
    if (!reads_level(u, j)) continue;
    __syncthreads();  // K region free
    {
      const T* U = nodes.at(bh, N, j, source_first(u, j), SZ);
      for (int idx = tid; idx < SZ / VEC; idx += NT) {
        const int p = idx / (DK / VEC), c = idx % (DK / VEC);
        *reinterpret_cast<V16*>(&u_s[p * LDK + c * VEC]) = *reinterpret_cast<const V16*>(U + idx * VEC);
      }
    }
    __syncthreads();
    const float wdec = rowok ? fast_exp2(cli + gap_of(gapv, j)) : 0.f;
    float yd = 0.f;
#pragma unroll
    for (int mt = 0; mt < MTV; ++mt) {
      f32x4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KSK; ++ks)
        t = M::mma(M::load(&u_s[(mt * 16 + r16) * LDK + ks * M::KSTEP + g * M::KPL]), qf[ks], t);
#pragma unroll
      for (int r = 0; r < 4; ++r) yd += t[r] * dorl[mt][r];
    }
    yd = sum_over_groups(yd);
    if (g == 0 && rowok) dl_s[i * L + LOG2R + j] = wdec * yd;
    const float sc = rowok ? wdec * lrow[LOG2R + j] : 0.f;
#pragma unroll
    for (int mt = 0; mt < MTK; ++mt) {
      f32x4 t = {0.f, 0.f, 0.f, 0.f};
      if constexpr (M::KPL == 8) {
#pragma unroll
        for (int st = 0; st < DV / 32; ++st)
          t = M::mma(frag_rows<T>(u_s, LDK, 32 * st, 16 * mt, 0), pack_rl(dorl[2 * st], dorl[2 * st + 1]), t);
      } else {
#pragma unroll
        for (int tt = 0; tt < MTV; ++tt)
#pragma unroll
          for (int r = 0; r < 4; ++r) t = M::mma(frag_rows<T>(u_s, LDK, 16 * tt, 16 * mt, r), dorl[tt][r], t);
      }
      acc[mt] += sc * t;
    }
  }

  // ---- outputs: dq (row i, d_k entries 16 mt + 4 g + r), q . dq, dlambda rows
  float qd = 0.f;
#pragma unroll
  for (int mt = 0; mt < MTK; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t e = qrow * DK + 16 * mt + 4 * g + r;
      if (rowok) {
        dq[e] = from_f32<T>(acc[mt][r]);
        qd += acc[mt][r] * to_f32(q[qkrow * DK + 16 * mt + 4 * g + r]);
      }
    }
  qd = sum_over_groups(qd);
  if (g == 0 && rowok) qdq[qrow] = qd;
  __syncthreads();
  for (int idx = tid; idx < nrow * L; idx += NT) {
    const int r = idx / L, l = idx % L;
    dlam[((row0 + r) * H + h) * L + l] = dl_s[idx];
  }
}

// ---------------------------------------------------------------------------------------------
// k_bwd_dkv: one workgroup of R/16 waves per (b, h, tile); wave w owns key rows 16 w .. 16 w + 15,
// one per MFMA column.  Q and dO of the tile resident in LDS.
//   intra: S = Q K^T and G = dO V^T per 16-query tile (queries >= keys), weights from the query's
//          lambda row; dk^T += Q^T (w (.) G), dv^T += dO^T (w (.) S);
//   inter: per key-side level, D_j copied into LDS: dk^T += w' D_j^T V^T, dv^T += w' D_j K^T;
//   then dcum = q . dq - k . dk per row, summed from each row to the tile end into dlog_alpha,
//   and the tile's total into tsum.
// ---------------------------------------------------------------------------------------------
template <typename T, int C, int DK, int DV>
__global__ __launch_bounds__(4 * tile_rows(C)) void k_bwd_dkv(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v, const T* __restrict__ dout,
    const float* __restrict__ log_alpha, const float* __restrict__ lam, RevNodes<T> rev, const float* __restrict__ qdq,
    T* __restrict__ dk, T* __restrict__ dv, float* __restrict__ dla, float* __restrict__ tsum, int64_t Tlen, int H,
    int Hqk, int L, int J) {
  using M = Mfma<T>;
  typedef typename Vec16<T>::type V16;
  constexpr int R = tile_rows(C), NW = R / 16, NT = 64 * NW;
  constexpr int VEC = Vec16<T>::N;
  constexpr int LDQ = DK + 16, LDO = DV + 16;
  constexpr int KSK = DK / M::KSTEP, KSV = DV / M::KSTEP, MTK = DK / 16, MTV = DV / 16;
  constexpr int SZ = DK * DV;
  static_assert(DV <= R, "a summary fits in the Q region");
  __shared__ T q_s[R * LDQ];
  __shared__ T o_s[R * LDO];
  __shared__ float cl_s[R];
  __shared__ float wsum_s[4];
  __shared__ float lam_s[R * kMaxLevels];
  __shared__ float dc_s[R];
  T* d_s = q_s;

  const int64_t N = (Tlen + R - 1) / R;
  const int64_t work = xcd_remap(blockIdx.x, (int64_t)gridDim.x);  // logical order (b, h, u)
  const int u = (int)(work % N);
  const int64_t bh = work / N;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t row0 = (int64_t)b * Tlen + (int64_t)u * R;
  const int nrow = (int)((Tlen - (int64_t)u * R) < R ? (Tlen - (int64_t)u * R) : R);
  const int jk = 16 * wave + r16;  // this lane's key row
  const bool keyok = jk < nrow;
  const int64_t krow = (row0 + (keyok ? jk : 0)) * H + h;
  const int hq = h / (H / Hqk);  // this head's query/key head
  const int64_t kqrow = (row0 + (keyok ? jk : 0)) * Hqk + hq;

  const float la = tile_gate<R>(log_alpha, row0, nrow, H, h);
  load_tile<T, DK, LDQ, R, NT>(q_s, q, row0, nrow, Hqk, hq);
  load_tile<T, DV, LDO, R, NT>(o_s, dout, row0, nrow, H, h);
  load_lambda<NT>(lam_s, lam, row0, nrow, H, h, L);

  typename M::frag kf[KSK], vf[KSV];
#pragma unroll
  for (int ks = 0; ks < KSK; ++ks)
    kf[ks] = keyok ? M::load(k + kqrow * DK + ks * M::KSTEP + g * M::KPL) : typename M::frag{};
#pragma unroll
  for (int ks = 0; ks < KSV; ++ks)
    vf[ks] = keyok ? M::load(v + krow * DV + ks * M::KSTEP + g * M::KPL) : typename M::frag{};
  f32x4 vrl[MTV];  // v of key row jk at d_v entries 16 mt + 4 g + r
#pragma unroll
  for (int mt = 0; mt < MTV; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) vrl[mt][r] = keyok ? to_f32(v[krow * DV + 16 * mt + 4 * g + r]) : 0.f;

  tile_cumsum_of<R>(la, nrow, cl_s, wsum_s);
  const float clj = cl_s[jk];

  f32x4 ak[MTK], av[MTV];
#pragma unroll
  for (int mt = 0; mt < MTK; ++mt) ak[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int mt = 0; mt < MTV; ++mt) av[mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // weights of one 16-query tile QT >= wave, result layout (query 16 QT + 4 g + r, key jk)
  auto query_tile = [&](int QT, f32x4& wg, f32x4& wp) {
    f32x4 s = {0.f, 0.f, 0.f, 0.f}, gg = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KSK; ++ks)
      s = M::mma(M::load(&q_s[(QT * 16 + r16) * LDQ + ks * M::KSTEP + g * M::KPL]), kf[ks], s);
#pragma unroll
    for (int ks = 0; ks < KSV; ++ks)
      gg = M::mma(M::load(&o_s[(QT * 16 + r16) * LDO + ks * M::KSTEP + g * M::KPL]), vf[ks], gg);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int ii = 16 * QT + 4 * g + r;
      const bool ok = ii >= jk && ii < nrow && keyok;
      const int lv = QT > wave ? level_local(16 * QT, 16 * wave) : level_local(ii, jk);
      const float lw = ok ? lam_s[ii * L + lv] * fast_exp2(cl_s[ii] - clj) : 0.f;
      wg[r] = lw * gg[r];
      wp[r] = lw * s[r];
    }
  };

  if constexpr (M::KPL == 8) {
    for (int st = wave / 2; st < NW / 2; ++st) {
      f32x4 g0 = {0.f, 0.f, 0.f, 0.f}, p0 = g0, g1, p1;
      if (2 * st >= wave) query_tile(2 * st, g0, p0);
      query_tile(2 * st + 1, g1, p1);
      const bf16x8 bg = pack_rl(g0, g1), bq = pack_rl(p0, p1);
#pragma unroll
      for (int mt = 0; mt < MTK; ++mt) ak[mt] = M::mma(frag_rows<T>(q_s, LDQ, 32 * st, 16 * mt, 0), bg, ak[mt]);
#pragma unroll
      for (int mt = 0; mt < MTV; ++mt) av[mt] = M::mma(frag_rows<T>(o_s, LDO, 32 * st, 16 * mt, 0), bq, av[mt]);
    }
  } else {
    for (int QT = wave; QT < NW; ++QT) {
      f32x4 g0, p0;
      query_tile(QT, g0, p0);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
#pragma unroll
        for (int mt = 0; mt < MTK; ++mt) ak[mt] = M::mma(frag_rows<T>(q_s, LDQ, 16 * QT, 16 * mt, r), g0[r], ak[mt]);
#pragma unroll
        for (int mt = 0; mt < MTV; ++mt) av[mt] = M::mma(frag_rows<T>(o_s, LDO, 16 * QT, 16 * mt, r), p0[r], av[mt]);
      }
    }
  }

  // ---- key-side levels: gap'_j (lane j - 1) is the exclusive sum over the lower key-side levels
  float gapr;
  {
    const int jl = lane + 1;
    float t = 0.f;
    if (jl <= J && key_level(u, jl, N)) t = rev.dtot[rev.slot(bh, jl, (int64_t)u >> jl)];
    gapr = wave_inclusive_scan(t) - t;
  }
  const float tot_u = cl_s[R - 1];
  for (int j = 1; j <= J; ++j) {
    if (!key_level(u, j, N)) continue;
    __syncthreads();  // Q region free
    {
      const T* D = rev.d + rev.slot(bh, j, (int64_t)u >> j) * SZ;
      for (int idx = tid; idx < SZ / VEC; idx += NT) {
        const int p = idx / (DK / VEC), c = idx % (DK / VEC);
        *reinterpret_cast<V16*>(&d_s[p * LDQ + c * VEC]) = *reinterpret_cast<const V16*>(D + idx * VEC);
      }
    }
    __syncthreads();
    const float wk = keyok ? fast_exp2(tot_u - clj + gap_of(gapr, j)) : 0.f;
    // dk^T[n][jk] += wk sum_p D[p][n] v[p]
#pragma unroll
    for (int mt = 0; mt < MTK; ++mt) {
      f32x4 t = {0.f, 0.f, 0.f, 0.f};
      if constexpr (M::KPL == 8) {
#pragma unroll
        for (int st = 0; st < DV / 32; ++st)
          t = M::mma(frag_rows<T>(d_s, LDQ, 32 * st, 16 * mt, 0), pack_rl(vrl[2 * st], vrl[2 * st + 1]), t);
      } else {
#pragma unroll
        for (int tt = 0; tt < MTV; ++tt)
#pragma unroll
          for (int r = 0; r < 4; ++r) t = M::mma(frag_rows<T>(d_s, LDQ, 16 * tt, 16 * mt, r), vrl[tt][r], t);
      }
      ak[mt] += wk * t;
    }
    // dv^T[p][jk] += wk sum_n D[p][n] k[n]
#pragma unroll
    for (int mt = 0; mt < MTV; ++mt) {
      f32x4 t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KSK; ++ks)
        t = M::mma(M::load(&d_s[(mt * 16 + r16) * LDQ + ks * M::KSTEP + g * M::KPL]), kf[ks], t);
      av[mt] += wk * t;
    }
  }

  // ---- outputs
  float kd = 0.f;
#pragma unroll
  for (int mt = 0; mt < MTK; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t e = krow * DK + 16 * mt + 4 * g + r;
      if (keyok) {
        dk[e] = from_f32<T>(ak[mt][r]);
        kd += ak[mt][r] * to_f32(k[kqrow * DK + 16 * mt + 4 * g + r]);
      }
    }
#pragma unroll
  for (int mt = 0; mt < MTV; ++mt)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (keyok) dv[krow * DV + 16 * mt + 4 * g + r] = from_f32<T>(av[mt][r]);
  kd = sum_over_groups(kd);
  if (g == 0) dc_s[jk] = keyok ? qdq[krow] - kd : 0.f;
  __syncthreads();
  // suffix sums of dcum within the tile: thread x < R (whole waves) scans row R - 1 - x
  const int row = R - 1 - tid;
  float x = 0.f;
  if (tid < R) x = wave_inclusive_scan(dc_s[row]);
  if (tid < R && lane == 63) wsum_s[wave] = x;
  __syncthreads();
  if (tid < R) {
    for (int w = 0; w < wave; ++w) x += wsum_s[w];
    if (row < nrow) dla[(row0 + row) * H + h] = x;
    if (tid == R - 1) tsum[bh * N + u] = x;
  }
}

// ---------------------------------------------------------------------------------------------
// bf16 tiles of 128 rows (C = 64).  The tile's two operand tiles and the level summaries live in
// swizzled LDS tiles filled by direct global->LDS loads; 4 waves, wave w owning the 16-row groups
// w and 7 - w (equal causal work, and every LDS fragment feeds two MFMAs).  The inter-tile levels
// run first, their summaries alternating between the two tile regions, the next one copied in
// while the current one is used; the operand tiles are copied in behind the last level, and the
// intra-tile part runs last.
// ---------------------------------------------------------------------------------------------
constexpr int kBwdFastThreads = 256;
constexpr int kBwdFastRows = 128;

namespace {

// dO-style operand of one row in the result-row k order: slots 0-3 = x[32 st + 4 g + 0..3],
// slots 4-7 = x[32 st + 16 + 4 g + 0..3] (pairs with frag_down_rows_swz reads of k rows 32 st ..).
__device__ inline bf16x8 load_rl_pair(const __bf16* row, int st) {
  const int g = (threadIdx.x & 63) >> 4;
  const bf16x4 lo = *reinterpret_cast<const bf16x4*>(row + 32 * st + 4 * g);
  const bf16x4 hi = *reinterpret_cast<const bf16x4*>(row + 32 * st + 16 + 4 * g);
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

}  // namespace

template <int DK, int DV>
__global__ __launch_bounds__(kBwdFastThreads, 2) void k_bwd_dq_fast(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    const __bf16* __restrict__ dout, const float* __restrict__ lam, Nodes<__bf16> nodes, __bf16* __restrict__ dq,
    float* __restrict__ dlam, float* __restrict__ qdq, int64_t Tlen, int H, int Hqk, int L, int J) {
  using M = Mfma<__bf16>;
  typedef __bf16 bf;
  typedef typename M::frag frag;
  constexpr int R = kBwdFastRows, LOG2R = 7, NT = kBwdFastThreads;
  constexpr int KSK = DK / 32, KSV = DV / 32, MTK = DK / 16, MTV = DV / 16;
  constexpr int SZ = DK * DV;
  static_assert(DK <= R && DV <= R, "a summary fits in either tile region");
  __shared__ bf k_s[R * DK];
  __shared__ bf v_s[R * DV];
  __shared__ float lam_s[R * kMaxLevels];
  __shared__ float cl_s[R];

  const int64_t N = (Tlen + R - 1) / R;
  const int64_t work = xcd_remap(blockIdx.x, (int64_t)gridDim.x);  // logical order (b, h, u)
  const int u = (int)(work % N);
  const int64_t bh = work / N;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t row0 = (int64_t)b * Tlen + (int64_t)u * R;
  const int nrow = (int)((Tlen - (int64_t)u * R) < R ? (Tlen - (int64_t)u * R) : R);
  const int gA = wave, gB = 7 - wave;            // this wave's 16-row groups
  const int iA = 16 * gA + r16, iB = 16 * gB + r16;
  const bool liveB = 16 * gB < nrow;             // nrow is a multiple of C = 64; group A is always live
  const int hq = h / (H / Hqk);                  // this head's query/key head

  // ---- loads: gates and lambda into LDS, this lane's rows of q and dO into registers, the first
  //      level's summary (or, without levels, the K and V tiles) into the K region
  lds_gather4<NT>(cl_s, R, [&](int x) { return nodes.cl + (bh * N + u) * R + x; });
  lds_copy_lambda<R, NT>(lam_s, lam, row0, H, h, L, nrow);
  frag qA[KSK], qB[KSK], dA[KSV], dB[KSV], pA[KSV], pB[KSV];
  {
    const int rB = iB < nrow ? iB : nrow - 1;
    const bf* qa = q + ((row0 + iA) * Hqk + hq) * DK;
    const bf* qb = q + ((row0 + rB) * Hqk + hq) * DK;
    const bf* da = dout + ((row0 + iA) * H + h) * DV;
    const bf* db = dout + ((row0 + rB) * H + h) * DV;
#pragma unroll
    for (int ks = 0; ks < KSK; ++ks) {
      qA[ks] = M::load(qa + ks * 32 + g * 8);
      qB[ks] = M::load(qb + ks * 32 + g * 8);
    }
#pragma unroll
    for (int ks = 0; ks < KSV; ++ks) {
      dA[ks] = M::load(da + ks * 32 + g * 8);
      dB[ks] = M::load(db + ks * 32 + g * 8);
      pA[ks] = load_rl_pair(da, ks);
      pB[ks] = load_rl_pair(db, ks);
    }
  }
  auto copy_tile = [&](bf* region) {
    if (region == k_s) lds_copy_rows<DK, R, NT>(k_s, k + (row0 * Hqk + hq) * DK, (int64_t)Hqk * DK, nrow);
    else lds_copy_rows<DV, R, NT>(v_s, v + (row0 * H + h) * DV, (int64_t)H * DV, nrow);
  };
  auto next_level = [&](int j) {
    for (++j; j <= J; ++j)
      if (reads_level(u, j)) return j;
    return 0;
  };
  // the first summary (or the tile) is requested before the gaps are summed: their sum waits for
  // every load issued before it
  int j = next_level(0);
  if (j) lds_copy_rows<DK, DV, NT>(k_s, nodes.at(bh, N, j, source_first(u, j), SZ), DK, DV);
  else {
    copy_tile(k_s);
    copy_tile(v_s);
  }
  const float gapv = level_gaps(nodes, bh, N, u, J);
  if (!liveB) {
#pragma unroll
    for (int ks = 0; ks < KSK; ++ks) qB[ks] = frag{};
#pragma unroll
    for (int ks = 0; ks < KSV; ++ks) dB[ks] = pB[ks] = frag{};
  }
  const float* lrowA = &lam_s[iA * kMaxLevels];
  const float* lrowB = &lam_s[(liveB ? iB : 0) * kMaxLevels];
  const int64_t growA = (row0 + iA) * H + h, growB = (row0 + (liveB ? iB : 0)) * H + h;

  f32x4 accA[MTK], accB[MTK];
#pragma unroll
  for (int mt = 0; mt < MTK; ++mt) accA[mt] = accB[mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // One inter-tile level from `cur`; the next level's summary (or, after the last level, the
  // operand tile of that region) goes to `nxt`.
  auto level_step = [&](const bf* cur, bf* nxt) {
    wait_vmem();
    __syncthreads();  // `cur` complete and visible; every wave is done with `nxt`
    const int jn = next_level(j);
    if (jn) lds_copy_rows<DK, DV, NT>(nxt, nodes.at(bh, N, jn, source_first(u, jn), SZ), DK, DV);
    else copy_tile(nxt);
    const float gap = gap_of(gapv, j);
    const float wA = fast_exp2(cl_s[iA] + gap), wB = liveB ? fast_exp2(cl_s[iB] + gap) : 0.f;
    // y^T = U Q^T, dlambda = dO . y
    float yA = 0.f, yB = 0.f;
#pragma unroll
    for (int mt = 0; mt < MTV; ++mt) {
      f32x4 tA = {0.f, 0.f, 0.f, 0.f}, tB = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KSK; ++ks) {
        const frag uf = frag_along_row_swz<DK>(cur, 16 * mt, 4 * ks);
        tA = M::mma(uf, qA[ks], tA);
        tB = M::mma(uf, qB[ks], tB);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        yA += tA[r] * static_cast<float>(pA[mt >> 1][(mt & 1) * 4 + r]);
        yB += tB[r] * static_cast<float>(pB[mt >> 1][(mt & 1) * 4 + r]);
      }
    }
    yA = sum_over_groups(yA);
    yB = sum_over_groups(yB);
    // dq^T += lambda w U^T dO^T.  lambda^(7 + j) of these rows is read here for the last time: its
    // LDS slot takes dlambda^(7 + j) (each row is read and written by its own wave only).
    const float sA = wA * lrowA[LOG2R + j], sB = liveB ? wB * lrowB[LOG2R + j] : 0.f;
    if (g == 0) {
      lam_s[iA * kMaxLevels + LOG2R + j] = wA * yA;
      if (liveB) lam_s[iB * kMaxLevels + LOG2R + j] = wB * yB;
    }
#pragma unroll
    for (int mt = 0; mt < MTK; ++mt) {
      f32x4 tA = {0.f, 0.f, 0.f, 0.f}, tB = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < KSV; ++st) {
        const frag uf = frag_down_rows_swz<DK>(cur, 32 * st, 16 * mt);
        tA = M::mma(uf, pA[st], tA);
        tB = M::mma(uf, pB[st], tB);
      }
      accA[mt] += sA * tA;
      accB[mt] += sB * tB;
    }
    j = jn;
  };
  if (j) {
    bf* cur = k_s;
    bf* nxt = v_s;
    while (true) {
      level_step(cur, nxt);
      if (!j) break;
      bf* t = cur;
      cur = nxt;
      nxt = t;
    }
    __syncthreads();  // every wave is done with the last summary
    copy_tile(cur);
  }
  wait_vmem();
  __syncthreads();  // K and V tiles (and gates, lambda) visible

  // ---- intra-tile: key tiles 2 st, 2 st + 1 per step
  const float cliA = cl_s[iA], cliB = cl_s[iB];
  float dlA[LOG2R + 1], dlB[LOG2R + 1];
#pragma unroll
  for (int l = 0; l <= LOG2R; ++l) dlA[l] = dlB[l] = 0.f;
  auto key_tile = [&](int KT, int gX, int iX, float cliX, const float* lrowX, const frag* kf, const frag* vf,
                      const frag* qX, const frag* dX, f32x4& wg, float (&dl)[LOG2R + 1]) {
    f32x4 s = {0.f, 0.f, 0.f, 0.f}, gg = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KSK; ++ks) s = M::mma(kf[ks], qX[ks], s);
#pragma unroll
    for (int ks = 0; ks < KSV; ++ks) gg = M::mma(vf[ks], dX[ks], gg);
    if (KT < gX) {
      const int lv = level_local(16 * gX, 16 * KT);
      const float lw = lrowX[lv];
      float pg = 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float e = fast_exp2(cliX - cl_s[16 * KT + 4 * g + r]);
        pg += e * s[r] * gg[r];
        wg[r] = lw * e * gg[r];
      }
      add_level(dl, lv, pg);
    } else {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int jj = 16 * KT + 4 * g + r;
        const bool ok = jj <= iX;
        const int lv = level_local(iX, jj);
        const float e = ok ? fast_exp2(cliX - cl_s[jj]) : 0.f;
        add_level(dl, ok ? lv : 0, e * s[r] * gg[r]);
        wg[r] = ok ? lrowX[lv] * e * gg[r] : 0.f;
      }
    }
  };
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    const bool needA = 2 * st <= gA, needB = 2 * st <= gB && liveB;
    if (!needA && !needB) break;
    f32x4 wgA[2], wgB[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int KT = 2 * st + hh;
      wgA[hh] = wgB[hh] = f32x4{0.f, 0.f, 0.f, 0.f};
      const bool useA = KT <= gA, useB = KT <= gB && liveB;
      if (!useA && !useB) continue;
      frag kf[KSK], vf[KSV];
#pragma unroll
      for (int ks = 0; ks < KSK; ++ks) kf[ks] = frag_along_row_swz<DK>(k_s, 16 * KT, 4 * ks);
#pragma unroll
      for (int ks = 0; ks < KSV; ++ks) vf[ks] = frag_along_row_swz<DV>(v_s, 16 * KT, 4 * ks);
      if (useA) key_tile(KT, gA, iA, cliA, lrowA, kf, vf, qA, dA, wgA[hh], dlA);
      if (useB) key_tile(KT, gB, iB, cliB, lrowB, kf, vf, qB, dB, wgB[hh], dlB);
    }
    const bf16x8 bA = pack_rl(wgA[0], wgA[1]), bB = pack_rl(wgB[0], wgB[1]);
#pragma unroll
    for (int mt = 0; mt < MTK; ++mt) {
      const frag kd = frag_down_rows_swz<DK>(k_s, 32 * st, 16 * mt);
      if (needA) accA[mt] = M::mma(kd, bA, accA[mt]);
      if (needB) accB[mt] = M::mma(kd, bB, accB[mt]);
    }
  }

  // ---- dlambda of the intra-tile levels and zeros for the inter-tile levels this tile does not
  //      read go to the rows' lambda slots (the wave's own rows, no longer read), then every row
  //      leaves whole
#pragma unroll
  for (int l = 0; l <= LOG2R; ++l) {
    const float xA = sum_over_groups(dlA[l]), xB = sum_over_groups(dlB[l]);
    if (g == 0) {
      lam_s[iA * kMaxLevels + l] = xA;
      lam_s[iB * kMaxLevels + l] = xB;
    }
  }
  for (int jj = 1; LOG2R + jj < L; ++jj)
    if (jj > J || !reads_level(u, jj)) {
      if (g == 0) {
        lam_s[iA * kMaxLevels + LOG2R + jj] = 0.f;
        lam_s[iB * kMaxLevels + LOG2R + jj] = 0.f;
      }
    }

  // ---- q . dq (fp32 accumulators), then dq through LDS as whole rows
  float qdA = 0.f, qdB = 0.f;
  {
    const bf* qa = q + ((row0 + iA) * Hqk + hq) * DK + 4 * g;
    const bf* qb = q + ((row0 + (liveB ? iB : 0)) * Hqk + hq) * DK + 4 * g;
#pragma unroll
    for (int mt = 0; mt < MTK; ++mt) {
      const bf16x4 xa = *reinterpret_cast<const bf16x4*>(qa + 16 * mt);
      const bf16x4 xb = *reinterpret_cast<const bf16x4*>(qb + 16 * mt);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        qdA += accA[mt][r] * static_cast<float>(xa[r]);
        qdB += accB[mt][r] * static_cast<float>(xb[r]);
      }
    }
  }
  qdA = sum_over_groups(qdA);
  qdB = sum_over_groups(qdB);
  if (g == 0) {
    qdq[growA] = qdA;
    if (liveB) qdq[growB] = qdB;
  }
  __syncthreads();  // every wave is done with K
  auto stage_rows = [&](const f32x4* acc, int i) {
#pragma unroll
    for (int mt = 0; mt < MTK; ++mt) {
      bf16x4 val;
#pragma unroll
      for (int r = 0; r < 4; ++r) val[r] = static_cast<bf>(acc[mt][r]);
      *reinterpret_cast<bf16x4*>(k_s + swz<DK>(i, 2 * mt + (g >> 1)) + 4 * (g & 1)) = val;
    }
  };
  stage_rows(accA, iA);
  stage_rows(accB, iB);
  __syncthreads();
  for (int idx = tid; idx < nrow * L; idx += NT) {
    const int r = idx / L, l = idx % L;
    dlam[((row0 + r) * H + h) * L + l] = lam_s[r * kMaxLevels + l];
  }
  constexpr int OCH = DK / 8;
#pragma unroll
  for (int it = 0; it < R * OCH / NT; ++it) {
    const int idx = it * NT + tid, r = idx / OCH, c = idx % OCH;
    if (r < nrow)
      *reinterpret_cast<bf16x8*>(dq + ((row0 + r) * H + h) * DK + 8 * c) =
          *reinterpret_cast<const bf16x8*>(k_s + swz<DK>(r, c));
  }
}

template <int DK, int DV>
__global__ __launch_bounds__(kBwdFastThreads, 2) void k_bwd_dkv_fast(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    const __bf16* __restrict__ dout, const float* __restrict__ lam, Nodes<__bf16> nodes, RevNodes<__bf16> rev,
    const float* __restrict__ qdq, __bf16* __restrict__ dk, __bf16* __restrict__ dv, float* __restrict__ dla,
    float* __restrict__ tsum, int64_t Tlen, int H, int Hqk, int L, int J) {
  using M = Mfma<__bf16>;
  typedef __bf16 bf;
  typedef typename M::frag frag;
  constexpr int R = kBwdFastRows, NT = kBwdFastThreads;
  constexpr int KSK = DK / 32, KSV = DV / 32, MTK = DK / 16, MTV = DV / 16;
  constexpr int SZ = DK * DV;
  static_assert(DK <= R && DV <= R, "a summary fits in either tile region");
  __shared__ bf q_s[R * DK];
  __shared__ bf o_s[R * DV];
  __shared__ float lam_s[R * kMaxLevels];
  __shared__ float cl_s[R];
  __shared__ float dc_s[R];
  __shared__ float wsum_s[2];

  const int64_t N = (Tlen + R - 1) / R;
  const int64_t work = xcd_remap(blockIdx.x, (int64_t)gridDim.x);  // logical order (b, h, u)
  const int u = (int)(work % N);
  const int64_t bh = work / N;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t row0 = (int64_t)b * Tlen + (int64_t)u * R;
  const int nrow = (int)((Tlen - (int64_t)u * R) < R ? (Tlen - (int64_t)u * R) : R);
  const int gA = wave, gB = 7 - wave;            // this wave's 16-key groups
  const int jA = 16 * gA + r16, jB = 16 * gB + r16;
  const bool liveB = 16 * gB < nrow;
  const int64_t growA = (row0 + jA) * H + h, growB = (row0 + (liveB ? jB : 0)) * H + h;
  const int hq = h / (H / Hqk);  // this head's query/key head
  const int64_t kqA = (row0 + jA) * Hqk + hq, kqB = (row0 + (liveB ? jB : 0)) * Hqk + hq;

  lds_gather4<NT>(cl_s, R, [&](int x) { return nodes.cl + (bh * N + u) * R + x; });
  lds_copy_lambda<R, NT>(lam_s, lam, row0, H, h, L, nrow);
  frag kA[KSK], kB[KSK], wA_[KSV], wB_[KSV];  // k rows (along d_k), v rows in the result-row k order
#pragma unroll
  for (int ks = 0; ks < KSK; ++ks) {
    kA[ks] = M::load(k + kqA * DK + ks * 32 + g * 8);
    kB[ks] = M::load(k + kqB * DK + ks * 32 + g * 8);
  }
#pragma unroll
  for (int st = 0; st < KSV; ++st) {
    wA_[st] = load_rl_pair(v + growA * DV, st);
    wB_[st] = load_rl_pair(v + growB * DV, st);
  }
  auto copy_tile = [&](bf* region) {
    if (region == q_s) lds_copy_rows<DK, R, NT>(q_s, q + (row0 * Hqk + hq) * DK, (int64_t)Hqk * DK, nrow);
    else lds_copy_rows<DV, R, NT>(o_s, dout + (row0 * H + h) * DV, (int64_t)H * DV, nrow);
  };
  auto next_level = [&](int j) {
    for (++j; j <= J; ++j)
      if (key_level(u, j, N)) return j;
    return 0;
  };
  // q . dq of this lane's key rows, for the tile's tail (loaded now, unconditionally: a load under a
  // lane condition is waited for where the branch ends)
  const float qdqA = qdq[growA], qdqB = qdq[growB];
  // the first key-side summary (or the tile) is requested before the gaps are summed: their sum
  // waits for every load issued before it
  int j = next_level(0);
  if (j) lds_copy_rows<DK, DV, NT>(q_s, rev.d + rev.slot(bh, j, (int64_t)u >> j) * SZ, DK, DV);
  else {
    copy_tile(q_s);
    copy_tile(o_s);
  }
  float gapr;
  {
    const int jl = lane + 1;
    const bool use = jl <= J && key_level(u, jl, N);
    const float tr = rev.dtot[rev.slot(bh, use ? jl : 1, use ? (int64_t)u >> jl : 0)];
    const float t = use ? tr : 0.f;
    gapr = wave_inclusive_scan(t) - t;
  }
  if (!liveB) {
#pragma unroll
    for (int ks = 0; ks < KSK; ++ks) kB[ks] = frag{};
#pragma unroll
    for (int st = 0; st < KSV; ++st) wB_[st] = frag{};
  }

  f32x4 akA[MTK], akB[MTK], avA[MTV], avB[MTV];
#pragma unroll
  for (int mt = 0; mt < MTK; ++mt) akA[mt] = akB[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int mt = 0; mt < MTV; ++mt) avA[mt] = avB[mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto level_step = [&](const bf* cur, bf* nxt) {
    wait_vmem();
    __syncthreads();
    const int jn = next_level(j);
    if (jn) lds_copy_rows<DK, DV, NT>(nxt, rev.d + rev.slot(bh, jn, (int64_t)u >> jn) * SZ, DK, DV);
    else copy_tile(nxt);
    // keys here are in a full tile (a later group exists): decay to the tile end, then the gap
    const float tot = cl_s[R - 1], gp = gap_of(gapr, j);
    const float wkA = fast_exp2(tot - cl_s[jA] + gp), wkB = liveB ? fast_exp2(tot - cl_s[jB] + gp) : 0.f;
    // dk^T[n][key] += w sum_p D[p][n] v[key][p]
#pragma unroll
    for (int mt = 0; mt < MTK; ++mt) {
      f32x4 tA = {0.f, 0.f, 0.f, 0.f}, tB = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < KSV; ++st) {
        const frag df = frag_down_rows_swz<DK>(cur, 32 * st, 16 * mt);
        tA = M::mma(df, wA_[st], tA);
        tB = M::mma(df, wB_[st], tB);
      }
      akA[mt] += wkA * tA;
      akB[mt] += wkB * tB;
    }
    // dv^T[p][key] += w sum_n D[p][n] k[key][n]
#pragma unroll
    for (int mt = 0; mt < MTV; ++mt) {
      f32x4 tA = {0.f, 0.f, 0.f, 0.f}, tB = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KSK; ++ks) {
        const frag df = frag_along_row_swz<DK>(cur, 16 * mt, 4 * ks);
        tA = M::mma(df, kA[ks], tA);
        tB = M::mma(df, kB[ks], tB);
      }
      avA[mt] += wkA * tA;
      avB[mt] += wkB * tB;
    }
    j = jn;
  };
  if (j) {
    bf* cur = q_s;
    bf* nxt = o_s;
    while (true) {
      level_step(cur, nxt);
      if (!j) break;
      bf* t = cur;
      cur = nxt;
      nxt = t;
    }
    __syncthreads();
    copy_tile(cur);
  }
  // v rows along d_v for the intra-tile G (the result-row order copies are no longer needed)
  frag vA[KSV], vB[KSV];
#pragma unroll
  for (int ks = 0; ks < KSV; ++ks) {
    vA[ks] = M::load(v + growA * DV + ks * 32 + g * 8);
    vB[ks] = liveB ? M::load(v + growB * DV + ks * 32 + g * 8) : frag{};
  }
  wait_vmem();
  __syncthreads();  // Q and dO tiles visible

  // ---- intra-tile: query tiles 2 st, 2 st + 1 per step (queries at or after the keys)
  const float clA = cl_s[jA], clB = cl_s[jB];
  // weights of query tile QT for one key group from its S and G tiles (result layout: query
  // 16 QT + 4 g + r, key jX), into slots 4 hh + r of the packed B operands
  auto weights = [&](int QT, int gX, int jX, float clX, const f32x4& s, const f32x4& gg, bf16x8& bg, bf16x8& bp,
                     int hh) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * QT + 4 * g + r;
      const bool ok = (QT > gX || i >= jX) && i < nrow;
      const int lv = QT > gX ? level_local(16 * QT, 16 * gX) : level_local(i, jX);
      const float lw = ok ? lam_s[i * kMaxLevels + lv] * fast_exp2(cl_s[i] - clX) : 0.f;
      bg[4 * hh + r] = static_cast<bf>(lw * gg[r]);
      bp[4 * hh + r] = static_cast<bf>(lw * s[r]);
    }
  };
#pragma unroll
  for (int st = 0; st < 4; ++st) {
    const bool needA = 2 * st + 1 >= gA, needB = 2 * st + 1 >= gB && liveB;
    if (!needA && !needB) continue;
    bf16x8 bgA = {}, bpA = {}, bgB = {}, bpB = {};
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const int QT = 2 * st + hh;
      const bool useA = QT >= gA, useB = QT >= gB && liveB;
      if (!useA && !useB) continue;
      // S = Q K^T and G = dO V^T of this query tile for both key groups, one fragment at a time
      f32x4 sA = {0.f, 0.f, 0.f, 0.f}, sB = sA, gA_ = sA, gB_ = sA;
#pragma unroll
      for (int ks = 0; ks < KSK; ++ks) {
        const frag f = frag_along_row_swz<DK>(q_s, 16 * QT, 4 * ks);
        if (useA) sA = M::mma(f, kA[ks], sA);
        if (useB) sB = M::mma(f, kB[ks], sB);
      }
#pragma unroll
      for (int ks = 0; ks < KSV; ++ks) {
        const frag f = frag_along_row_swz<DV>(o_s, 16 * QT, 4 * ks);
        if (useA) gA_ = M::mma(f, vA[ks], gA_);
        if (useB) gB_ = M::mma(f, vB[ks], gB_);
      }
      if (useA) weights(QT, gA, jA, clA, sA, gA_, bgA, bpA, hh);
      if (useB) weights(QT, gB, jB, clB, sB, gB_, bgB, bpB, hh);
    }
#pragma unroll
    for (int mt = 0; mt < MTK; ++mt) {
      const frag qd = frag_down_rows_swz<DK>(q_s, 32 * st, 16 * mt);
      if (needA) akA[mt] = M::mma(qd, bgA, akA[mt]);
      if (needB) akB[mt] = M::mma(qd, bgB, akB[mt]);
    }
#pragma unroll
    for (int mt = 0; mt < MTV; ++mt) {
      const frag od = frag_down_rows_swz<DV>(o_s, 32 * st, 16 * mt);
      if (needA) avA[mt] = M::mma(od, bpA, avA[mt]);
      if (needB) avB[mt] = M::mma(od, bpB, avB[mt]);
    }
  }

  // ---- k . dk, dcum = q . dq - k . dk
  float kdA = 0.f, kdB = 0.f;
  {
    const bf* ka = k + kqA * DK + 4 * g;
    const bf* kb = k + kqB * DK + 4 * g;
#pragma unroll
    for (int mt = 0; mt < MTK; ++mt) {
      const bf16x4 xa = *reinterpret_cast<const bf16x4*>(ka + 16 * mt);
      const bf16x4 xb = *reinterpret_cast<const bf16x4*>(kb + 16 * mt);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        kdA += akA[mt][r] * static_cast<float>(xa[r]);
        kdB += akB[mt][r] * static_cast<float>(xb[r]);
      }
    }
  }
  kdA = sum_over_groups(kdA);
  kdB = sum_over_groups(kdB);
  if (g == 0) {
    dc_s[jA] = qdqA - kdA;
    dc_s[jB] = liveB ? qdqB - kdB : 0.f;
  }
  __syncthreads();  // every wave is done with Q and dO; dc visible
  // ---- dk and dv through LDS as whole rows
  auto stage_k = [&](const f32x4 (&acc)[MTK], int i) {
#pragma unroll
    for (int mt = 0; mt < MTK; ++mt) {
      bf16x4 val;
#pragma unroll
      for (int r = 0; r < 4; ++r) val[r] = static_cast<bf>(acc[mt][r]);
      *reinterpret_cast<bf16x4*>(q_s + swz<DK>(i, 2 * mt + (g >> 1)) + 4 * (g & 1)) = val;
    }
  };
  auto stage_v = [&](const f32x4 (&acc)[MTV], int i) {
#pragma unroll
    for (int mt = 0; mt < MTV; ++mt) {
      bf16x4 val;
#pragma unroll
      for (int r = 0; r < 4; ++r) val[r] = static_cast<bf>(acc[mt][r]);
      *reinterpret_cast<bf16x4*>(o_s + swz<DV>(i, 2 * mt + (g >> 1)) + 4 * (g & 1)) = val;
    }
  };
  stage_k(akA, jA);
  stage_k(akB, jB);
  stage_v(avA, jA);
  stage_v(avB, jB);
  // suffix sums of dcum within the tile: thread x < R (two waves) scans row R - 1 - x
  const int row = R - 1 - tid;
  float x = 0.f;
  if (tid < R) x = wave_inclusive_scan(dc_s[row]);
  if (tid < R && lane == 63) wsum_s[wave] = x;
  __syncthreads();
  if (tid < R) {
    if (wave == 1) x += wsum_s[0];
    if (row < nrow) dla[(row0 + row) * H + h] = x;
    if (tid == R - 1) tsum[bh * N + u] = x;
  }
#pragma unroll
  for (int it = 0; it < R * (DK / 8) / NT; ++it) {
    const int idx = it * NT + tid, r = idx / (DK / 8), c = idx % (DK / 8);
    if (r < nrow)
      *reinterpret_cast<bf16x8*>(dk + ((row0 + r) * H + h) * DK + 8 * c) =
          *reinterpret_cast<const bf16x8*>(q_s + swz<DK>(r, c));
  }
#pragma unroll
  for (int it = 0; it < R * (DV / 8) / NT; ++it) {
    const int idx = it * NT + tid, r = idx / (DV / 8), c = idx % (DV / 8);
    if (r < nrow)
      *reinterpret_cast<bf16x8*>(dv + ((row0 + r) * H + h) * DV + 8 * c) =
          *reinterpret_cast<const bf16x8*>(o_s + swz<DV>(r, c));
  }
}

// ---------------------------------------------------------------------------------------------
// k_bwd_dgate: grid (ceil(T / 256), B * H); adds to each row's tile-local suffix sum the totals
// of all later tiles of its sequence.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_bwd_dgate(const float* __restrict__ tsum, float* __restrict__ dla,
                                                   int64_t Tlen, int H, int R) {
  __shared__ float red_s[4];
  const int64_t N = (Tlen + R - 1) / R;
  const int64_t bh = blockIdx.y;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int64_t t0 = (int64_t)blockIdx.x * 256;
  const int64_t t1 = t0 + 255 < Tlen - 1 ? t0 + 255 : Tlen - 1;
  const int64_t ulast = t1 / R;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  float s = 0.f;
  for (int64_t x = ulast + 1 + tid; x < N; x += 256) s += tsum[bh * N + x];
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
  if (lane == 0) red_s[wave] = s;
  __syncthreads();
  const float after = red_s[0] + red_s[1] + red_s[2] + red_s[3];  // tiles after the last one here
  const int64_t t = t0 + tid;
  if (t < Tlen) {
    float add = after;
    for (int64_t x = t / R + 1; x <= ulast; ++x) add += tsum[bh * N + x];
    dla[((int64_t)b * Tlen + t) * H + h] += add;
  }
}

// ---------------------------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------------------------
// ---------------------------------------------------------------------------------------------
// k_group_sum: heads sharing one query/key head -- out[b, t, hq, :] = sum over the group's heads h
// of in[b, t, h, :] (fp32 sums of the per-head gradients).  grid (ceil(rows * Hqk * D / 256)).
// ---------------------------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_group_sum(const T* __restrict__ in, T* __restrict__ out, int64_t rows, int H,
                                                   int Hqk, int D) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= rows * Hqk * D) return;
  const int d = (int)(idx % D);
  const int64_t rq = idx / D;  // (row, hq)
  const int hq = (int)(rq % Hqk);
  const int64_t row = rq / Hqk;
  const int G = H / Hqk;
  const T* src = in + (row * H + (int64_t)hq * G) * D + d;
  float acc = 0.f;
  for (int x = 0; x < G; ++x) acc += to_f32(src[(int64_t)x * D]);
  out[idx] = from_f32<T>(acc);
}

int64_t mamba2_bwd_workspace(int64_t B, int64_t T, int64_t H, int64_t Hqk, int64_t dk, int64_t dv, int64_t C,
                             int64_t esize, BwdLayout* lay) {
  BwdLayout w{};
  int64_t cur = mamba2_workspace(B, T, H, dk, dv, C, esize, true, &w.fwd);
  // the forward run in this workspace may be the single-pass one, which leaves its summaries in
  // its own layout: the backward's regions start after both
  if (esize == 2 && mamba2_fused_supported(1, C, dk, dv, true)) {
    const int64_t fused = mamba2_fused_workspace(B, T, H, dk, dv, nullptr, true);
    if (cur < fused) cur = fused;
  }
  auto al = [](int64_t x) { return (x + 255) & ~int64_t(255); };
  const int64_t N = w.fwd.N, BH = B * H, SZ = dk * dv;
  const int J = w.fwd.J;
  w.NR = (N + kRegionTiles - 1) / kRegionTiles;
  w.nd = 0;
  for (int j = 1; j <= J; ++j) w.nd += RevNodes<float>::groups(N, j);
  w.npart = 0;
  for (int j = 5; j <= J; ++j) w.npart += RevNodes<float>::parts(w.NR, j);
  const int64_t nd1 = w.nd > 0 ? w.nd : 1, np1 = w.npart > 0 ? w.npart : 1;
  w.bad = cur; cur += al(4);
  w.d = cur; cur += al(BH * nd1 * SZ * esize);
  w.dtot = cur; cur += al(BH * nd1 * 4);
  w.part = cur; cur += al(BH * np1 * SZ * 4);
  w.qdq = cur; cur += al(B * T * H * 4);
  w.tsum = cur; cur += al(BH * N * 4);
  if (Hqk < H) {  // per-head dq and dk before the sum over each group of heads
    w.dqh = cur; cur += al(B * T * H * dk * esize);
    w.dkh = cur; cur += al(B * T * H * dk * esize);
  }
  w.total = cur;
  if (lay) *lay = w;
  return cur;
}

// Compares the workspace's summary tag with the tag of this call's inputs: *bad = 1 on a mismatch.
__global__ void k_check_tag(const uint64_t* tag, WsTag want, int* bad) {
  const int i = threadIdx.x;
  const bool diff = i < 12 && tag[i] != want.v[i];
  const bool any = __any(diff);
  if (i == 0) *bad = any ? 1 : 0;
}

// NaN-fills every gradient when *bad is set (the reused summaries belonged to other inputs).
template <typename T>
__global__ void k_poison_grads(const int* bad, T* dq, int64_t nq, T* dk, T* dv, int64_t nv, float* dla, int64_t na,
                               float* dlam, int64_t nl) {
  if (*bad == 0) return;
  const T tn = from_f32<T>(__builtin_nanf(""));
  const float fn = __builtin_nanf("");
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nq; i += stride) dq[i] = dk[i] = tn;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += stride) dv[i] = tn;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < na; i += stride) dla[i] = fn;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nl; i += stride) dlam[i] = fn;
}

// Stages (ev[i] recorded before stage i, ev[4] after the last): 0 the forward summaries (skipped
// when the workspace already holds them), 1 the key-side summaries, 2 dq and dlambda, 3 dk, dv and
// dlog_alpha.
template <typename T, int C, int DK, int DV>
hipError_t launch_mamba2_bwd(const Mamba2BwdArgs& a, hipStream_t st, hipEvent_t* ev) {
  constexpr int R = tile_rows(C), SZ = DK * DV;
  BwdLayout w;
  mamba2_bwd_workspace(a.B, a.T, a.H, a.Hqk, DK, DV, C, sizeof(T), &w);
  Nodes<T> nodes = mamba2_nodes<T>(w.fwd, a.workspace, true);
  char* base = static_cast<char*>(a.workspace);
  if (a.reuse_summaries && a.fused_fwd) {  // the single-pass forward's summaries, by tile
    FusedLayout fl;
    mamba2_fused_workspace(a.B, a.T, a.H, DK, DV, &fl, true);
    nodes.by_u = reinterpret_cast<T*>(base + fl.ubwd);
    nodes.bsum = reinterpret_cast<const float*>(base + fl.bsum);
    nodes.bstride = fl.stride;
    nodes.t1 = reinterpret_cast<const float*>(base + fl.t1);
    nodes.cl = reinterpret_cast<float*>(base + fl.cl);
  }
  RevNodes<T> rev;
  rev.d = reinterpret_cast<T*>(base + w.d);
  rev.dtot = reinterpret_cast<float*>(base + w.dtot);
  rev.part = reinterpret_cast<float*>(base + w.part);
  rev.N = w.fwd.N;
  rev.NR = w.NR;
  rev.nd = w.nd;
  rev.npart = w.npart;
  float* qdq = reinterpret_cast<float*>(base + w.qdq);
  float* tsum = reinterpret_cast<float*>(base + w.tsum);
  const int J = w.fwd.J;
  const int64_t BH = a.B * a.H;
  const bool grouped = a.Hqk < a.H;
  // per-head dq, dk: the outputs themselves, or scratch summed over each group of heads at the end
  T* dqh = grouped ? reinterpret_cast<T*>(base + w.dqh) : (T*)a.dq;
  T* dkh = grouped ? reinterpret_cast<T*>(base + w.dkh) : (T*)a.dk;

  Mamba2Args fa{};
  fa.q = a.q; fa.k = a.k; fa.v = a.v; fa.log_alpha = a.log_alpha; fa.lambda = a.lambda; fa.o = nullptr;
  fa.B = a.B; fa.T = a.T; fa.H = a.H; fa.dk = DK; fa.dv = DV; fa.C = C; fa.Hqk = a.Hqk; fa.L = a.L;
  fa.workspace = a.workspace;
  int* bad = reinterpret_cast<int*>(base + w.bad);
  if (ev) (void)hipEventRecord(ev[0], st);
  if (!a.reuse_summaries) {
    const hipError_t e = launch_mamba2_summaries<T, C, DK, DV>(fa, w.fwd, nodes, st, nullptr);
    if (e != hipSuccess) return e;
  } else {
    hipLaunchKernelGGL(k_check_tag, dim3(1), dim3(64), 0, st,
                       reinterpret_cast<const uint64_t*>(base + w.fwd.tag), mamba2_tag(fa, sizeof(T), true), bad);
  }
  if (ev) (void)hipEventRecord(ev[1], st);
  if (J >= 1) {
    const int items = 7 + (J > 3 ? J - 3 : 0);
    hipLaunchKernelGGL((k_rev_state<T, C, DK, DV>), dim3((unsigned)(BH * w.NR * items)), dim3(kRevThreads), 0, st,
                       (const T*)a.q, (const T*)a.dout, a.lambda, nodes, rev, a.T, (int)a.H, (int)a.Hqk, a.L, J,
                       items);
  }
  if (J >= 5) {
    int64_t ng = 0;
    for (int j = 5; j <= J; ++j) ng += RevNodes<T>::groups(w.fwd.N, j);
    hipLaunchKernelGGL((k_rev_reduce<T>), dim3((unsigned)((SZ + 1023) / 1024), (unsigned)ng, (unsigned)BH), dim3(256),
                       0, st, nodes, rev, J, SZ);
  }
  if (ev) (void)hipEventRecord(ev[2], st);
  const dim3 gtile((unsigned)(w.fwd.N * BH));
  constexpr bool kFast = std::is_same<T, __bf16>::value && R == kBwdFastRows;
  if constexpr (kFast)
    hipLaunchKernelGGL((k_bwd_dq_fast<DK, DV>), gtile, dim3(kBwdFastThreads), 0, st, (const T*)a.q, (const T*)a.k,
                       (const T*)a.v, (const T*)a.dout, a.lambda, nodes, dqh, a.dlambda, qdq, a.T, (int)a.H,
                       (int)a.Hqk, a.L, J);
  else
    hipLaunchKernelGGL((k_bwd_dq<T, C, DK, DV>), gtile, dim3(4 * R), 0, st, (const T*)a.q, (const T*)a.k,
                       (const T*)a.v, (const T*)a.dout, a.log_alpha, a.lambda, nodes, dqh, a.dlambda, qdq, a.T,
                       (int)a.H, (int)a.Hqk, a.L, J);
  if (ev) (void)hipEventRecord(ev[3], st);
  if constexpr (kFast)
    hipLaunchKernelGGL((k_bwd_dkv_fast<DK, DV>), gtile, dim3(kBwdFastThreads), 0, st, (const T*)a.q, (const T*)a.k,
                       (const T*)a.v, (const T*)a.dout, a.lambda, nodes, rev, (const float*)qdq, dkh, (T*)a.dv,
                       a.dlog_alpha, tsum, a.T, (int)a.H, (int)a.Hqk, a.L, J);
  else
    hipLaunchKernelGGL((k_bwd_dkv<T, C, DK, DV>), gtile, dim3(4 * R), 0, st, (const T*)a.q, (const T*)a.k,
                       (const T*)a.v, (const T*)a.dout, a.log_alpha, a.lambda, rev, (const float*)qdq, dkh,
                       (T*)a.dv, a.dlog_alpha, tsum, a.T, (int)a.H, (int)a.Hqk, a.L, J);
  hipLaunchKernelGGL(k_bwd_dgate, dim3((unsigned)((a.T + 255) / 256), (unsigned)BH), dim3(256), 0, st,
                     (const float*)tsum, a.dlog_alpha, a.T, (int)a.H, R);
  if (grouped) {
    const int64_t n = a.B * a.T * a.Hqk * DK;
    hipLaunchKernelGGL((k_group_sum<T>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, (const T*)dqh, (T*)a.dq,
                       a.B * a.T, (int)a.H, (int)a.Hqk, DK);
    hipLaunchKernelGGL((k_group_sum<T>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, (const T*)dkh, (T*)a.dk,
                       a.B * a.T, (int)a.H, (int)a.Hqk, DK);
  }
  if (a.reuse_summaries) {
    const int64_t nq = a.B * a.T * a.Hqk * DK, nv = a.B * a.T * a.H * DV, na = a.B * a.T * a.H;
    hipLaunchKernelGGL((k_poison_grads<T>), dim3(512), dim3(256), 0, st, (const int*)bad, (T*)a.dq, nq, (T*)a.dk,
                       (T*)a.dv, nv, a.dlog_alpha, na, a.dlambda, na * a.L);
  }
  if (ev) (void)hipEventRecord(ev[4], st);
  return hipGetLastError();
}

const BwdEntry* mamba2_bwd_table(int* n) {
#define LL_BWD_ENTRY(T, C, DK, DV) {std::is_same<T, float>::value ? 0 : 1, C, DK, DV, &launch_mamba2_bwd<T, C, DK, DV>},
  static const BwdEntry table[] = {LL_MAMBA2_SHAPES(LL_BWD_ENTRY)};
#undef LL_BWD_ENTRY
  *n = sizeof(table) / sizeof(table[0]);
  return table;
}

}  // namespace ll
