// Log-linear Mamba-2 and Gated DeltaNet decoding: one token per call, O(log t) state per head
// (Sec. 3.2).  The Mamba-2 step is described here, the Gated DeltaNet step at k_gdn_decode_step.
//
// Per (b, h) the state is the list of Fenwick level states S^(l) (d_v x d_k).  Token t (0-based)
// updates it as the recurrent form does: for t >= 1, with p = lssb(t), level p+1 receives the
// sum of levels 0..p, levels 1..p are emptied, higher levels carry over, and every carried or
// merged level is multiplied by alpha_t; then level 0 becomes v_t k_t^T.  The output is
// o_t = sum_l lambda_t^(l) S_t^(l) q_t (Eq. 3 read-out).
//
// Storage (one caller-owned buffer, carved by decode_layout):
//   S      [B*H][L][d_v][d_k] fp32   levels 1 .. L-1 (slot 0 unused), each kept as c_l * S_stored
//   scale  [2][B*H][L]        fp32   c_l, double-buffered by step parity (read t-1, write t)
//   f0     [2][B*H][d_v + d_k] fp32  level 0 in factored form, v and k of the previous token
// The decays are applied lazily through the per-level scales, so a step reads only the levels
// that are not empty (scale != 0) and writes only the merged level p+1: O(popcount) level reads
// and one level write per head instead of touching all L levels twice.
//
// Work split: grid (d_v / 16, B*H), 256 threads; thread (row r = tid / 16, part c = tid % 16)
// owns d_v row 16 blockIdx.x + r and d_k entries [c d_k/16, (c+1) d_k/16) of every level; row
// sums are reduced over the 16 lanes of the row.  Workgroups of one head share nothing but the
// double-buffered scale and f0 arrays, written only by workgroup x = 0 into the other parity.
#include <type_traits>

#include "../../include/libloglinear.h"
#include "ll_device.hpp"

namespace ll {

constexpr int kDecodeThreads = 256;
constexpr int kDecodeMaxLevels = 32;

struct DecodeLayout {
  int64_t S = 0, scale = 0, f0 = 0, total = 0;
};

DecodeLayout decode_layout(int64_t B, int64_t H, int64_t dk, int64_t dv, int64_t L) {
  auto al = [](int64_t x) { return (x + 255) & ~int64_t(255); };
  const int64_t BH = B * H;
  DecodeLayout d;
  int64_t cur = 0;
  d.S = cur; cur += al(BH * L * dv * dk * 4);
  d.scale = cur; cur += al(2 * BH * L * 4);
  d.f0 = cur; cur += al(2 * BH * (dv + dk) * 4);
  d.total = cur;
  return d;
}

template <typename T, int DK, int DV>
__global__ __launch_bounds__(kDecodeThreads) void k_decode_step(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v, const float* __restrict__ log_alpha,
    const float* __restrict__ lam, T* __restrict__ o, float* __restrict__ S, const float* __restrict__ scale_in,
    float* __restrict__ scale_out, const float* __restrict__ f0_in, float* __restrict__ f0_out, int64_t t, int p,
    int L) {
  constexpr int NPT = DK / 16;  // d_k entries per thread
  static_assert(DK % 16 == 0 && DV % 16 == 0, "whole 16-entry pieces");
  const int64_t bh = blockIdx.y;
  const int tid = threadIdx.x, r = tid >> 4, c = tid & 15;
  const int row = blockIdx.x * 16 + r;
  const int n0 = c * NPT;

  float qv[NPT], kv[NPT];
#pragma unroll
  for (int i = 0; i < NPT; ++i) {
    qv[i] = to_f32(q[bh * DK + n0 + i]);
    kv[i] = to_f32(k[bh * DK + n0 + i]);
  }
  const float vrow = to_f32(v[bh * DV + row]);
  const float alpha = expf(log_alpha[bh]);
  auto lam_of = [&](int l) { return lam ? lam[bh * L + l] : 1.f; };
  const float* cin = scale_in + bh * L;
  float* Sh = S + bh * (int64_t)L * DV * DK;
  auto level_row = [&](int l) { return Sh + ((int64_t)l * DV + row) * DK + n0; };

  float acc = 0.f;  // this thread's part of sum_l lambda_l S^(l) q for its row
  if (t > 0) {
    // level p+1 <- levels 0..p (level 0 from the previous token's factors)
    const float c0 = cin[0];
    const float vold = f0_in[bh * (DV + DK) + row];
    float m[NPT];
#pragma unroll
    for (int i = 0; i < NPT; ++i) m[i] = c0 * vold * f0_in[bh * (DV + DK) + DV + n0 + i];
    for (int l = 1; l <= p; ++l) {
      const float cl = cin[l];
      if (cl == 0.f) continue;
      const float* src = level_row(l);
#pragma unroll
      for (int i = 0; i < NPT; ++i) m[i] += cl * src[i];
    }
    float* dst = level_row(p + 1);
    float d = 0.f;
#pragma unroll
    for (int i = 0; i < NPT; ++i) {
      dst[i] = m[i];
      d += m[i] * qv[i];
    }
    acc += lam_of(p + 1) * alpha * d;
    // levels above p+1 carry over, decayed by alpha_t
    for (int l = p + 2; l < L; ++l) {
      const float cl = cin[l];
      if (cl == 0.f) continue;
      const float* src = level_row(l);
      float e = 0.f;
#pragma unroll
      for (int i = 0; i < NPT; ++i) e += src[i] * qv[i];
      acc += lam_of(l) * cl * alpha * e;
    }
  }
  // level 0 = v_t k_t^T: its contribution to the row is v_t[row] (k_t . q_t)
  float kq = 0.f;
#pragma unroll
  for (int i = 0; i < NPT; ++i) kq += kv[i] * qv[i];
#pragma unroll
  for (int off = 8; off > 0; off >>= 1) {
    acc += __shfl_xor(acc, off, 64);
    kq += __shfl_xor(kq, off, 64);
  }
  if (c == 0) o[bh * DV + row] = from_f32<T>(acc + lam_of(0) * vrow * kq);

  // next step's scales and level-0 factors (the other parity buffer)
  if (blockIdx.x == 0) {
    float* cout = scale_out + bh * L;
    for (int l = tid; l < L; l += kDecodeThreads) {
      float x;
      if (l == 0) x = 1.f;
      else if (t == 0) x = 0.f;
      else if (l <= p) x = 0.f;
      else if (l == p + 1) x = alpha;
      else x = cin[l] * alpha;
      cout[l] = x;
    }
    float* f = f0_out + bh * (DV + DK);
    for (int i = tid; i < DV; i += kDecodeThreads) f[i] = to_f32(v[bh * DV + i]);
    for (int i = tid; i < DK; i += kDecodeThreads) f[DV + i] = to_f32(k[bh * DK + i]);
  }
}

// ---------------------------------------------------------------------------------------------
// Log-linear Gated DeltaNet decoding.  The transition alpha_t (I - beta_t k_t k_t^T) is not a
// scalar, so every nonempty level is rewritten each step; it acts on each d_v row of a level on
// its own (row x -> alpha (x - beta (x . k) k)), which keeps the same row split as above.  After
// token t the nonempty levels >= 1 are those l with bit l-1 of t set; for t >= 1 the lowest,
// p + 1 (p = lssb(t)), is the sum of the previous step's levels 0 .. p.  The output reads every
// level after its transition:
//   o_t = lambda^(0) beta_t (k_t . q_t) v_t + sum_l lambda^(l) alpha_t (S^(l) q_t - beta_t (k_t . q_t) S^(l) k_t),
// S^(l) being the level before the transition.  Storage as above; f0 holds beta v and k of the
// previous token (level 0, factored); the scales are not used.
// ---------------------------------------------------------------------------------------------
template <typename T, int DK, int DV>
__global__ __launch_bounds__(kDecodeThreads) void k_gdn_decode_step(
    const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v, const float* __restrict__ log_alpha,
    const float* __restrict__ beta, const float* __restrict__ lam, T* __restrict__ o, float* __restrict__ S,
    const float* __restrict__ f0_in, float* __restrict__ f0_out, int64_t t, int p, int L) {
  constexpr int NPT = DK / 16;
  static_assert(DK % 16 == 0 && DV % 16 == 0, "whole 16-entry pieces");
  const int64_t bh = blockIdx.y;
  const int tid = threadIdx.x, r = tid >> 4, c = tid & 15;
  const int row = blockIdx.x * 16 + r;
  const int n0 = c * NPT;
  // sum over the 16 lanes of a row (every lane receives it)
  auto row_sum = [](float x) {
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
  };

  float qv[NPT], kv[NPT];
#pragma unroll
  for (int i = 0; i < NPT; ++i) {
    qv[i] = to_f32(q[bh * DK + n0 + i]);
    kv[i] = to_f32(k[bh * DK + n0 + i]);
  }
  const float vrow = to_f32(v[bh * DV + row]);
  const float alpha = expf(log_alpha[bh]), bt = beta[bh];
  auto lam_of = [&](int l) { return lam ? lam[bh * L + l] : 1.f; };
  float* Sh = S + bh * (int64_t)L * DV * DK;
  auto level_row = [&](int l) { return Sh + ((int64_t)l * DV + row) * DK + n0; };
  float kq = 0.f;
#pragma unroll
  for (int i = 0; i < NPT; ++i) kq += kv[i] * qv[i];
  kq = row_sum(kq);

  float acc = 0.f;  // the row's output (identical in the row's 16 lanes)
  // transition of one level row x (this thread's part), written to dst, and its output term
  auto step_level = [&](float (&x)[NPT], float* dst, int l) {
    float a = 0.f, b = 0.f;
#pragma unroll
    for (int i = 0; i < NPT; ++i) {
      a += x[i] * kv[i];
      b += x[i] * qv[i];
    }
    a = row_sum(a);
    b = row_sum(b);
#pragma unroll
    for (int i = 0; i < NPT; ++i) dst[i] = alpha * (x[i] - bt * a * kv[i]);
    acc += lam_of(l) * alpha * (b - bt * kq * a);
  };
  if (t > 0) {
    // level p+1 <- previous levels 0 .. p (level 0 from the previous token's factors)
    const float* f = f0_in + bh * (DV + DK);
    const float bv = f[row];
    float m[NPT];
#pragma unroll
    for (int i = 0; i < NPT; ++i) m[i] = bv * f[DV + n0 + i];
    for (int l = 1; l <= p; ++l) {
      const float* src = level_row(l);
#pragma unroll
      for (int i = 0; i < NPT; ++i) m[i] += src[i];
    }
    step_level(m, level_row(p + 1), p + 1);
    // the other nonempty levels (bits above p of t) carry over, transitioned in place; their
    // rows are loaded kBatch levels at a time before any is processed (independent loads)
    constexpr int kBatch = 4;
    int64_t rest = t >> (p + 1);  // bit i: level p + 2 + i is nonempty
    int l0 = p + 2;
    while (rest) {
      int lv[kBatch];
      int n = 0;
      while (rest && n < kBatch) {
        const int sh = __builtin_ctzll((unsigned long long)rest);
        lv[n++] = l0 + sh;
        rest >>= sh + 1;
        l0 += sh + 1;
      }
      float x[kBatch][NPT];
#pragma unroll
      for (int b = 0; b < kBatch; ++b)
        if (b < n) {
          const float* src = level_row(lv[b]);
#pragma unroll
          for (int i = 0; i < NPT; ++i) x[b][i] = src[i];
        }
#pragma unroll
      for (int b = 0; b < kBatch; ++b)
        if (b < n) step_level(x[b], level_row(lv[b]), lv[b]);
    }
  }
  // level 0 = beta_t v_t k_t^T: its term is beta_t v_t[row] (k_t . q_t)
  if (c == 0) o[bh * DV + row] = from_f32<T>(acc + lam_of(0) * bt * vrow * kq);

  if (blockIdx.x == 0) {
    float* f = f0_out + bh * (DV + DK);
    for (int i = tid; i < DV; i += kDecodeThreads) f[i] = bt * to_f32(v[bh * DV + i]);
    for (int i = tid; i < DK; i += kDecodeThreads) f[DV + i] = to_f32(k[bh * DK + i]);
  }
}

// Zero-fills n floats (the decode state before its first token).
__global__ void k_zero_f32(float* __restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = 0.f;
}

template <typename T, int DK, int DV>
hipError_t launch_decode(const void* q, const void* k, const void* v, const float* log_alpha, const float* lambda,
                         void* o, void* state, int64_t t, int64_t B, int64_t H, int L, hipStream_t st) {
  const DecodeLayout d = decode_layout(B, H, DK, DV, L);
  char* base = static_cast<char*>(state);
  const int64_t BH = B * H;
  float* S = reinterpret_cast<float*>(base + d.S);
  float* scale = reinterpret_cast<float*>(base + d.scale);
  float* f0 = reinterpret_cast<float*>(base + d.f0);
  const int par = (int)(t & 1);
  const int p = t > 0 ? __builtin_ctzll((unsigned long long)t) : 0;
  hipLaunchKernelGGL((k_decode_step<T, DK, DV>), dim3(DV / 16, (unsigned)BH), dim3(kDecodeThreads), 0, st,
                     (const T*)q, (const T*)k, (const T*)v, log_alpha, lambda, (T*)o, S,
                     scale + (1 - par) * BH * L, scale + par * BH * L, f0 + (1 - par) * BH * (DV + DK),
                     f0 + par * BH * (DV + DK), t, p, L);
  return hipGetLastError();
}

template <typename T, int DK, int DV>
hipError_t launch_gdn_decode(const void* q, const void* k, const void* v, const float* log_alpha, const float* beta,
                             const float* lambda, void* o, void* state, int64_t t, int64_t B, int64_t H, int L,
                             hipStream_t st) {
  const DecodeLayout d = decode_layout(B, H, DK, DV, L);
  char* base = static_cast<char*>(state);
  const int64_t BH = B * H;
  float* S = reinterpret_cast<float*>(base + d.S);
  float* f0 = reinterpret_cast<float*>(base + d.f0);
  const int par = (int)(t & 1);
  const int p = t > 0 ? __builtin_ctzll((unsigned long long)t) : 0;
  hipLaunchKernelGGL((k_gdn_decode_step<T, DK, DV>), dim3(DV / 16, (unsigned)BH), dim3(kDecodeThreads), 0, st,
                     (const T*)q, (const T*)k, (const T*)v, log_alpha, beta, lambda, (T*)o, S,
                     f0 + (1 - par) * BH * (DV + DK), f0 + par * BH * (DV + DK), t, p, L);
  return hipGetLastError();
}

hipError_t launch_decode_init(void* state, int64_t B, int64_t H, int64_t dk, int64_t dv, int L, hipStream_t st) {
  const DecodeLayout d = decode_layout(B, H, dk, dv, L);
  // the scales and level-0 factors of both parities; the level data is read only where a
  // scale is nonzero, so it needs no clearing
  float* p = reinterpret_cast<float*>(static_cast<char*>(state) + d.scale);
  const int64_t n = (d.total - d.scale) / 4;
  hipLaunchKernelGGL(k_zero_f32, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p, n);
  return hipGetLastError();
}

typedef hipError_t (*DecodeLaunch)(const void*, const void*, const void*, const float*, const float*, void*, void*,
                                   int64_t, int64_t, int64_t, int, hipStream_t);
typedef hipError_t (*GdnDecodeLaunch)(const void*, const void*, const void*, const float*, const float*, const float*,
                                      void*, void*, int64_t, int64_t, int64_t, int, hipStream_t);
struct DecodeEntry {
  int dtype, dk, dv;
  DecodeLaunch launch;
  GdnDecodeLaunch gdn_launch;
};

#define LL_DECODE_SHAPES(X) \
  X(float, 16, 16)          \
  X(float, 64, 64)          \
  X(__bf16, 64, 64)         \
  X(__bf16, 128, 64)        \
  X(__bf16, 128, 128)

const DecodeEntry* decode_table(int* n) {
#define LL_ENTRY(T, DK, DV) \
  {std::is_same<T, float>::value ? 0 : 1, DK, DV, &launch_decode<T, DK, DV>, &launch_gdn_decode<T, DK, DV>},
  static const DecodeEntry table[] = {LL_DECODE_SHAPES(LL_ENTRY)};
#undef LL_ENTRY
  *n = sizeof(table) / sizeof(table[0]);
  return table;
}

}  // namespace ll

namespace {
const ll::DecodeEntry* find_decode(int32_t dtype, int64_t dk, int64_t dv) {
  int n = 0;
  const ll::DecodeEntry* t = ll::decode_table(&n);
  for (int i = 0; i < n; ++i)
    if (t[i].dtype == dtype && t[i].dk == dk && t[i].dv == dv) return &t[i];
  return nullptr;
}

ll_status check_decode(int64_t B, int64_t H, int64_t d_k, int64_t d_v, int32_t L, int32_t dtype) {
  if (B < 1 || H < 1 || d_k < 1 || d_v < 1 || L < 1) return LL_ERR_BAD_SHAPE;
  if (dtype != LL_F32 && dtype != LL_BF16) return LL_ERR_UNSUPPORTED;
  if (L > ll::kDecodeMaxLevels || B * H > 65535 || !find_decode(dtype, d_k, d_v)) return LL_ERR_UNSUPPORTED;
  return LL_OK;
}
}  // namespace

extern "C" {

size_t ll_decode_state_bytes(int64_t B, int64_t H, int64_t d_k, int64_t d_v, int32_t L) {
  if (B < 1 || H < 1 || d_k < 1 || d_v < 1 || L < 1) return 0;
  return (size_t)ll::decode_layout(B, H, d_k, d_v, L).total;
}

ll_status ll_mamba2_decode_init(void* state, size_t state_bytes, int64_t B, int64_t H, int64_t d_k, int64_t d_v,
                                int32_t L, int32_t dtype, void* stream) {
  if (!state) return LL_ERR_NULL_ARG;
  const ll_status s = check_decode(B, H, d_k, d_v, L, dtype);
  if (s != LL_OK) return s;
  if (state_bytes < (size_t)ll::decode_layout(B, H, d_k, d_v, L).total ||
      (reinterpret_cast<uintptr_t>(state) & 255))
    return LL_ERR_WORKSPACE;
  return ll::launch_decode_init(state, B, H, d_k, d_v, L, static_cast<hipStream_t>(stream)) == hipSuccess
             ? LL_OK
             : LL_ERR_HIP;
}

ll_status ll_mamba2_decode_step(const void* q, const void* k, const void* v, const float* log_alpha,
                                const float* lambda, void* o, void* state, size_t state_bytes, int64_t t, int64_t B,
                                int64_t H, int64_t d_k, int64_t d_v, int32_t L, int32_t dtype, void* stream) {
  if (!q || !k || !v || !log_alpha || !o || !state) return LL_ERR_NULL_ARG;
  const ll_status s = check_decode(B, H, d_k, d_v, L, dtype);
  if (s != LL_OK) return s;
  // token t needs level lssb(t) + 1 < L, i.e. t < 2^(L-1)
  if (t < 0 || (L - 1 < 62 && t >= (int64_t(1) << (L - 1)))) return LL_ERR_BAD_SHAPE;
  if (state_bytes < (size_t)ll::decode_layout(B, H, d_k, d_v, L).total ||
      (reinterpret_cast<uintptr_t>(state) & 255))
    return LL_ERR_WORKSPACE;
  const ll::DecodeEntry* e = find_decode(dtype, d_k, d_v);
  return e->launch(q, k, v, log_alpha, lambda, o, state, t, B, H, L, static_cast<hipStream_t>(stream)) == hipSuccess
             ? LL_OK
             : LL_ERR_HIP;
}

ll_status ll_gdn_decode_init(void* state, size_t state_bytes, int64_t B, int64_t H, int64_t d_k, int64_t d_v,
                             int32_t L, int32_t dtype, void* stream) {
  return ll_mamba2_decode_init(state, state_bytes, B, H, d_k, d_v, L, dtype, stream);
}

ll_status ll_gdn_decode_step(const void* q, const void* k, const void* v, const float* log_alpha, const float* beta,
                             const float* lambda, void* o, void* state, size_t state_bytes, int64_t t, int64_t B,
                             int64_t H, int64_t d_k, int64_t d_v, int32_t L, int32_t dtype, void* stream) {
  if (!q || !k || !v || !log_alpha || !beta || !o || !state) return LL_ERR_NULL_ARG;
  const ll_status s = check_decode(B, H, d_k, d_v, L, dtype);
  if (s != LL_OK) return s;
  if (t < 0 || (L - 1 < 62 && t >= (int64_t(1) << (L - 1)))) return LL_ERR_BAD_SHAPE;
  if (state_bytes < (size_t)ll::decode_layout(B, H, d_k, d_v, L).total ||
      (reinterpret_cast<uintptr_t>(state) & 255))
    return LL_ERR_WORKSPACE;
  const ll::DecodeEntry* e = find_decode(dtype, d_k, d_v);
  return e->gdn_launch(q, k, v, log_alpha, beta, lambda, o, state, t, B, H, L, static_cast<hipStream_t>(stream)) ==
                 hipSuccess
             ? LL_OK
             : LL_ERR_HIP;
}

}  // extern "C"
