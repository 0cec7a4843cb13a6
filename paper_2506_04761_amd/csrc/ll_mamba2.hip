// Log-linear Mamba-2 forward: O = (Q K^T (.) M^S (.) M^H) V  (Sec. 3.4), computed with the
// chunkwise algorithm of Sec. 3.3 (Eq. 5) in three kernels:
//
//   chunk_state  per chunk z: chunk-local cumulative log-gate cl, total tot_z, and the chunk
//                state S_z = sum_t exp(tot_z - cl_t) v_t k_t^T  (d_v x d_k, MFMA, K = C tokens).
//   level_scan   per (b, h), elementwise over state entries, sequential over chunks: the
//                summary of every source group each inter-chunk level reads (decayed to the
//                group end), plus the decay gap from a group's end to each reader chunk.
//                With lambda == NULL: the single running state entering every chunk.
//   chunk_out    per chunk: the intra-chunk C x C masked contraction (the block-diagonal D of
//                Eq. 5) and, for every set bit j-1 of the chunk index, the lambda-weighted
//                inter-chunk term  lambda_t^(log2 C + j) exp(cl_t + gap) q_t^T U_j  (the
//                masked Q S update of the chunkwise algorithm, App. C Alg. 1).
//
// Decays are kept in the log2 domain (gates pre-multiplied by log2 e) and every exp2 argument
// is <= 0: chunk-local cumulative sums and exact range sums of chunk totals, never differences
// of sequence-long prefix sums.
#include <type_traits>

#include "ll_device.hpp"
#include "ll_launch.hpp"

namespace ll {

// ---------------------------------------------------------------------------------------------
// Kernel 1: chunk states.  One workgroup (4 waves) per (chunk, head, batch).
// ---------------------------------------------------------------------------------------------
template <typename T, int C, int DK, int DV>
__global__ __launch_bounds__(256) void k_chunk_state(const T* __restrict__ k, const T* __restrict__ v,
                                                     const float* __restrict__ log_alpha,
                                                     float* __restrict__ states, float* __restrict__ tot2_out,
                                                     int64_t Tlen, int H) {
  using M = Mfma<T>;
  constexpr int VEC = Vec16<T>::N;
  constexpr int PAD = VEC;          // keeps 16-lane row accesses on distinct LDS banks
  constexpr int LDT = C + PAD;      // row stride of the transposed tiles (elements)
  __shared__ T vt_s[DV * LDT];      // V^T  [p][t]
  __shared__ T kt_s[DK * LDT];      // (decay * K)^T  [n][t]
  __shared__ float dec_s[C];

  const int z = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t N = Tlen / C;
  const int64_t tok0 = (int64_t)b * Tlen + (int64_t)z * C;  // first token row of the chunk

  if (wave == 0) {
    float la = lane < C ? log_alpha[(tok0 + lane) * H + h] * kLog2e : 0.f;
    float cl = wave_inclusive_scan(la);
    float tot = __shfl(cl, C - 1, 64);
    if (lane < C) dec_s[lane] = exp2f(tot - cl);
    if (lane == 0) tot2_out[((int64_t)b * H + h) * N + z] = tot;
  }
  __syncthreads();

  // Stage V^T and (dec * K)^T.
  for (int idx = tid; idx < C * DV / VEC; idx += 256) {
    const int t = idx / (DV / VEC), d0 = (idx % (DV / VEC)) * VEC;
    typename Vec16<T>::type x = *reinterpret_cast<const typename Vec16<T>::type*>(v + ((tok0 + t) * H + h) * DV + d0);
#pragma unroll
    for (int e = 0; e < VEC; ++e) vt_s[(d0 + e) * LDT + t] = x[e];
  }
  for (int idx = tid; idx < C * DK / VEC; idx += 256) {
    const int t = idx / (DK / VEC), d0 = (idx % (DK / VEC)) * VEC;
    typename Vec16<T>::type x = *reinterpret_cast<const typename Vec16<T>::type*>(k + ((tok0 + t) * H + h) * DK + d0);
    const float dt = dec_s[t];
#pragma unroll
    for (int e = 0; e < VEC; ++e) kt_s[(d0 + e) * LDT + t] = from_f32<T>(to_f32(x[e]) * dt);
  }
  __syncthreads();

  // S^T[p][n] = sum_t V^T[p][t] (dec K)^T[n][t]:  M = p, N = n, K = t.
  constexpr int MT = DV / 16, NT = DK / 16;
  float* out = states + (((int64_t)b * H + h) * N + z) * (int64_t)(DV * DK);
  const int r16 = lane & 15, g = lane >> 4;
  for (int tile = wave; tile < MT * NT; tile += 4) {
    const int mt = tile / NT, nt = tile % NT;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < C / M::KSTEP; ++ks) {
      const int k0 = ks * M::KSTEP + g * M::KPL;
      acc = M::mma(M::load(&vt_s[(mt * 16 + r16) * LDT + k0]), M::load(&kt_s[(nt * 16 + r16) * LDT + k0]), acc);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) out[(int64_t)(mt * 16 + 4 * g + r) * DK + nt * 16 + r16] = acc[r];
  }
}

// ---------------------------------------------------------------------------------------------
// Kernel 2: level scan.  Elementwise over the d_v*d_k state entries (4 per thread), sequential
// over the chunks of one (b, h).
//
// Level j (group size 2^(j-1) chunks): the source groups are the even-indexed groups; inside
// one, acc_j <- exp2(tot_z) acc_j + S_z, reset at the group start; at the group end the
// summary (all chunk states decayed to the group end) is stored if some chunk reads it.
// gap_j(z) = sum of tot over the chunks of z's own aligned 2^(j-1)-block that precede z.
// ---------------------------------------------------------------------------------------------
constexpr int kMaxLevels = 24;  // inter-chunk levels: supports T/C up to 2^24

template <typename TN>
__global__ __launch_bounds__(256) void k_level_scan(const float* __restrict__ states,
                                                    const float* __restrict__ tot2, TN* __restrict__ nodes,
                                                    float* __restrict__ gaps2, int64_t N, int J, int SZ,
                                                    int64_t nodes_per_bh, int has_lambda) {
  const int64_t bh = blockIdx.y;
  const int e0 = (blockIdx.x * 256 + threadIdx.x) * 4;
  const float* tot = tot2 + bh * N;

  if (blockIdx.x == 0 && threadIdx.x == 0 && has_lambda) {
    float gsum[kMaxLevels];
#pragma unroll
    for (int j = 0; j < kMaxLevels; ++j) gsum[j] = 0.f;
    for (int64_t z = 0; z < N; ++z) {
      const float tz = tot[z];
#pragma unroll
      for (int j = 1; j <= kMaxLevels; ++j) {
        if (j <= J) {
          if ((z & ((int64_t(1) << (j - 1)) - 1)) == 0) gsum[j - 1] = 0.f;
          gaps2[(bh * N + z) * J + (j - 1)] = gsum[j - 1];
          gsum[j - 1] += tz;
        }
      }
    }
  }
  if (e0 >= SZ) return;

  const float* src = states + bh * N * SZ + e0;
  TN* dst = nodes + bh * nodes_per_bh * SZ + e0;
  if (!has_lambda) {
    f32x4 run = {0.f, 0.f, 0.f, 0.f};
    for (int64_t z = 0; z < N; ++z) {
      const f32x4 s = *reinterpret_cast<const f32x4*>(src + z * SZ);
      const float e = exp2f(tot[z]);
#pragma unroll
      for (int c = 0; c < 4; ++c) dst[z * SZ + c] = from_f32<TN>(run[c]);
      run = run * e + s;
    }
    return;
  }
  f32x4 acc[kMaxLevels];
#pragma unroll
  for (int j = 0; j < kMaxLevels; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  f32x4 s_next = *reinterpret_cast<const f32x4*>(src);
  for (int64_t z = 0; z < N; ++z) {
    const f32x4 s = s_next;
    if (z + 1 < N) s_next = *reinterpret_cast<const f32x4*>(src + (z + 1) * SZ);
    const float e = exp2f(tot[z]);
#pragma unroll
    for (int j = 1; j <= kMaxLevels; ++j) {
      const int64_t m = z >> (j - 1);
      if (j > J || (m & 1)) continue;                       // beyond the top level, or z reads
      const int64_t mask = (int64_t(1) << (j - 1)) - 1;
      if ((z & mask) == 0) acc[j - 1] = s;                   // group start
      else acc[j - 1] = acc[j - 1] * e + s;
      if (((z + 1) & mask) == 0 && ((m + 1) << (j - 1)) < N) {  // group end with a reader
        TN* d = dst + node_slot(N, j, m << (j - 1)) * SZ;
#pragma unroll
        for (int c = 0; c < 4; ++c) d[c] = from_f32<TN>(acc[j - 1][c]);
      }
    }
  }
}

// ---------------------------------------------------------------------------------------------
// Kernel 3: chunk outputs.  One wave per (chunk, head, batch).
//
// Orientation: the wave builds O^T (d_v x C) so that the query index is the MFMA column:
//   S^T = K Q^T        (keys x queries, K = d_k),  masked in registers,
//   O^T += V^T P^T     (P^T in the result layout of S^T is directly a B operand once its k
//                       slots are matched by loading V^T at the same keys),
//   O^T += w (.) U^T Q^T  per inter-chunk level, w = per-query weight (a column scale).
// ---------------------------------------------------------------------------------------------
template <typename T, int C, int DK, int DV, bool HAS_LAMBDA>
__global__ __launch_bounds__(64) void k_chunk_out(const T* __restrict__ q, const T* __restrict__ k,
                                                  const T* __restrict__ v, const float* __restrict__ log_alpha,
                                                  const float* __restrict__ lam, const T* __restrict__ nodes,
                                                  const float* __restrict__ gaps2, T* __restrict__ o,
                                                  int64_t Tlen, int H, int L, int J, int64_t nodes_per_bh) {
  using M = Mfma<T>;
  constexpr int VEC = Vec16<T>::N;
  constexpr int LDK = DK + VEC;   // K row stride (elements)
  constexpr int LDV = C + VEC;    // V^T row stride (elements)
  constexpr int LDL = 24;         // lambda row stride in LDS (>= L for every supported T)
  constexpr int QT = C / 16, MT = DV / 16, KS = DK / M::KSTEP;
  constexpr int LOG2C = (C == 16) ? 4 : (C == 32) ? 5 : (C == 64) ? 6 : 7;
  __shared__ T k_s[C * LDK];
  __shared__ T vt_s[DV * LDV];
  __shared__ float cl_s[C];
  __shared__ float lam_s[HAS_LAMBDA ? C * LDL : 1];

  const int z = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int lane = threadIdx.x, r16 = lane & 15, g = lane >> 4;
  const int64_t N = Tlen / C;
  const int64_t bh = (int64_t)b * H + h;
  const int64_t tok0 = (int64_t)b * Tlen + (int64_t)z * C;

  {
    float la = lane < C ? log_alpha[(tok0 + lane) * H + h] * kLog2e : 0.f;
    float cl = wave_inclusive_scan(la);
    if (lane < C) cl_s[lane] = cl;
  }
  if constexpr (HAS_LAMBDA) {
    for (int idx = lane; idx < C * L; idx += 64) {
      const int t = idx / L, l = idx % L;
      lam_s[t * LDL + l] = lam[((tok0 + t) * H + h) * L + l];
    }
  }
  for (int idx = lane; idx < C * DK / VEC; idx += 64) {
    const int t = idx / (DK / VEC), d0 = (idx % (DK / VEC)) * VEC;
    *reinterpret_cast<typename Vec16<T>::type*>(&k_s[t * LDK + d0]) =
        *reinterpret_cast<const typename Vec16<T>::type*>(k + ((tok0 + t) * H + h) * DK + d0);
  }
  for (int idx = lane; idx < C * DV / VEC; idx += 64) {
    const int t = idx / (DV / VEC), d0 = (idx % (DV / VEC)) * VEC;
    typename Vec16<T>::type x = *reinterpret_cast<const typename Vec16<T>::type*>(v + ((tok0 + t) * H + h) * DV + d0);
#pragma unroll
    for (int e = 0; e < VEC; ++e) vt_s[(d0 + e) * LDV + t] = x[e];
  }

  // Q^T fragments (B operand), kept in registers for the whole chunk.
  typename M::frag qf[QT][KS];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[qt][ks] = M::load(q + ((tok0 + qt * 16 + r16) * H + h) * DK + ks * M::KSTEP + g * M::KPL);
  __syncthreads();

  f32x4 oacc[MT][QT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) oacc[mt][qt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // ---- intra-chunk stage: D of Eq. 5
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int i = qt * 16 + r16;      // this lane's query (chunk-local)
    const float cli = cl_s[i];
    f32x4 p[QT];
#pragma unroll
    for (int kt = 0; kt <= qt; ++kt) {
      f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        s = M::mma(M::load(&k_s[(kt * 16 + r16) * LDK + ks * M::KSTEP + g * M::KPL]), qf[qt][ks], s);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = kt * 16 + 4 * g + r;  // key (chunk-local)
        float w = 0.f;
        if (j <= i) {
          w = exp2f(cli - cl_s[j]);
          if constexpr (HAS_LAMBDA) w *= lam_s[i * LDL + level_local(i, j)];
        }
        p[kt][r] = s[r] * w;
      }
    }
#pragma unroll
    for (int kt = qt + 1; kt < QT; ++kt) p[kt] = f32x4{0.f, 0.f, 0.f, 0.f};

    if constexpr (M::KPL == 8) {
      // bf16: one k step = 32 keys = key tiles (2 ks, 2 ks + 1); slots 0-3 <- tile 2 ks rows
      // 4g..4g+3, slots 4-7 <- tile 2 ks + 1 rows 4g..4g+3.
#pragma unroll
      for (int ks = 0; ks < (QT + 1) / 2; ++ks) {
        if (2 * ks > qt) break;
        typename M::frag bp;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          bp[r] = from_f32<T>(p[2 * ks][r]);
          bp[4 + r] = (2 * ks + 1 < QT) ? from_f32<T>(p[2 * ks + 1][r]) : from_f32<T>(0.f);
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const T* row = &vt_s[(mt * 16 + r16) * LDV + ks * 32 + 4 * g];
          const bf16x4 lo = *reinterpret_cast<const bf16x4*>(row);
          const bf16x4 hi = *reinterpret_cast<const bf16x4*>(row + 16);
          const typename M::frag a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          oacc[mt][qt] = M::mma(a, bp, oacc[mt][qt]);
        }
      }
    } else {
      // fp32: one k step = 4 keys {kt*16 + 4g + r : g}, i.e. slot r of every lane group.
#pragma unroll
      for (int kt = 0; kt <= qt; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
            oacc[mt][qt] = M::mma(vt_s[(mt * 16 + r16) * LDV + kt * 16 + 4 * g + r], p[kt][r], oacc[mt][qt]);
    }
  }

  // ---- inter-chunk stage
  if constexpr (HAS_LAMBDA) {
    for (int j = 1; j <= J; ++j) {
      if (!reads_level(z, j)) continue;
      const T* U = nodes + (bh * nodes_per_bh + node_slot(N, j, source_first(z, j))) * (int64_t)(DV * DK);
      const float gap = gaps2[(bh * N + z) * J + (j - 1)];
      float w[QT];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        const int i = qt * 16 + r16;
        w[qt] = lam_s[i * LDL + LOG2C + j] * exp2f(cl_s[i] + gap);
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        f32x4 tmp[QT];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) tmp[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const typename M::frag a = M::load(U + (mt * 16 + r16) * DK + ks * M::KSTEP + g * M::KPL);
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) tmp[qt] = M::mma(a, qf[qt][ks], tmp[qt]);
        }
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) oacc[mt][qt] += w[qt] * tmp[qt];
      }
    }
  } else {
    if (z > 0) {
      const T* U = nodes + (bh * nodes_per_bh + z) * (int64_t)(DV * DK);
      float w[QT];
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) w[qt] = exp2f(cl_s[qt * 16 + r16]);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        f32x4 tmp[QT];
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) tmp[qt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const typename M::frag a = M::load(U + (mt * 16 + r16) * DK + ks * M::KSTEP + g * M::KPL);
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) tmp[qt] = M::mma(a, qf[qt][ks], tmp[qt]);
        }
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) oacc[mt][qt] += w[qt] * tmp[qt];
      }
    }
  }

  // ---- store O: lane holds query qt*16 + r16, d_v entries mt*16 + 4g .. +3
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    T* orow = o + ((tok0 + qt * 16 + r16) * H + h) * DV + 4 * g;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) orow[mt * 16 + r] = from_f32<T>(oacc[mt][qt][r]);
  }
}

// ---------------------------------------------------------------------------------------------
// Debug level map: the level each (t, s) pair receives from the device functions above.
// ---------------------------------------------------------------------------------------------
__global__ void k_debug_level_map(int64_t Tlen, int C, int log2C, int J, int8_t* out) {
  const int64_t t = blockIdx.x;
  for (int64_t s = threadIdx.x; s < Tlen; s += blockDim.x) {
    int lev = -1;
    if (s <= t) {
      const int64_t zt = t / C, zs = s / C;
      if (zt == zs) {
        lev = level_local(int(t % C), int(s % C));
      } else {
        lev = -2;  // no source group claims the pair: a bug
        for (int j = 1; j <= J; ++j)
          if (reads_level(zt, j) && zs >= source_first(zt, j) && zs < source_first(zt, j) + (int64_t(1) << (j - 1)))
            lev = log2C + j;
      }
    }
    out[t * Tlen + s] = (int8_t)lev;
  }
}

// ---------------------------------------------------------------------------------------------
// Host-side launchers
// ---------------------------------------------------------------------------------------------
// Enqueues the three stages on `st`.  With `ev` non-null, ev[i] is recorded before stage i
// and ev[3] after the last one (used by the timed entry point).
template <typename T, int C, int DK, int DV>
hipError_t launch_mamba2(const Mamba2Args& a, hipStream_t st, hipEvent_t* ev) {
  const int64_t N = a.T / C;
  const int SZ = DK * DV;
  dim3 grid((unsigned)N, (unsigned)a.H, (unsigned)a.B);
  if (ev) (void)hipEventRecord(ev[0], st);
  hipLaunchKernelGGL((k_chunk_state<T, C, DK, DV>), grid, dim3(256), 0, st, (const T*)a.k, (const T*)a.v,
                     a.log_alpha, a.ws.states, a.ws.tot2, a.T, (int)a.H);
  if (ev) (void)hipEventRecord(ev[1], st);
  dim3 grid2((unsigned)((SZ / 4 + 255) / 256), (unsigned)(a.B * a.H));
  hipLaunchKernelGGL((k_level_scan<T>), grid2, dim3(256), 0, st, a.ws.states, a.ws.tot2, (T*)a.ws.nodes,
                     a.ws.gaps2, N, a.J, SZ, a.ws.nodes_per_bh, a.lambda != nullptr ? 1 : 0);
  if (ev) (void)hipEventRecord(ev[2], st);
  if (a.lambda)
    hipLaunchKernelGGL((k_chunk_out<T, C, DK, DV, true>), grid, dim3(64), 0, st, (const T*)a.q, (const T*)a.k,
                       (const T*)a.v, a.log_alpha, a.lambda, (const T*)a.ws.nodes, a.ws.gaps2, (T*)a.o, a.T,
                       (int)a.H, a.L, a.J, a.ws.nodes_per_bh);
  else
    hipLaunchKernelGGL((k_chunk_out<T, C, DK, DV, false>), grid, dim3(64), 0, st, (const T*)a.q, (const T*)a.k,
                       (const T*)a.v, a.log_alpha, a.lambda, (const T*)a.ws.nodes, a.ws.gaps2, (T*)a.o, a.T,
                       (int)a.H, a.L, a.J, a.ws.nodes_per_bh);
  if (ev) (void)hipEventRecord(ev[3], st);
  return hipGetLastError();
}

hipError_t launch_debug_level_map(int64_t T, int C, int log2C, int J, int8_t* out, hipStream_t st) {
  hipLaunchKernelGGL(k_debug_level_map, dim3((unsigned)T), dim3(256), 0, st, T, C, log2C, J, out);
  return hipGetLastError();
}

#define LL_MAMBA2_SHAPES(X)        \
  X(float, 16, 16, 16)             \
  X(float, 64, 64, 64)             \
  X(__bf16, 64, 64, 64)            \
  X(__bf16, 64, 128, 64)           \
  X(__bf16, 64, 128, 128)

const KernelEntry* mamba2_table(int* n) {
#define LL_ENTRY(T, C, DK, DV) {std::is_same<T, float>::value ? 0 : 1, C, DK, DV, &launch_mamba2<T, C, DK, DV>},
  static const KernelEntry table[] = {LL_MAMBA2_SHAPES(LL_ENTRY)};
#undef LL_ENTRY
  *n = sizeof(table) / sizeof(table[0]);
  return table;
}

}  // namespace ll
