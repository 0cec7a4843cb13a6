// C ABI of libloglinear: argument validation, workspace carving and kernel dispatch.
// All checks run on the host before anything is enqueued.
#include <atomic>
#include <mutex>
#include <type_traits>

#include "../../include/libloglinear.h"
#include "ll_launch.hpp"

namespace {

constexpr int kMaxL = 24;          // lambda levels the kernels stage (T <= 2^23)
constexpr int64_t kMaxTiles = 8192; // tiles per sequence (the running scan stages their totals in LDS)

inline int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }
inline bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }
inline int bitlen64(uint64_t x) { return x ? 64 - __builtin_clzll(x) : 0; }
inline int64_t elem_size(int32_t dtype) { return dtype == LL_BF16 ? 2 : 4; }

int32_t levels_of(int64_t T) { return T < 1 ? -1 : (T == 1 ? 1 : bitlen64(uint64_t(T - 1)) + 1); }

const ll::KernelEntry* find_mamba2(int32_t dtype, int64_t C, int64_t dk, int64_t dv) {
  int n = 0;
  const ll::KernelEntry* t = ll::mamba2_table(&n);
  for (int i = 0; i < n; ++i)
    if (t[i].dtype == dtype && t[i].C == C && t[i].dk == dk && t[i].dv == dv) return &t[i];
  return nullptr;
}

const ll::BwdEntry* find_mamba2_bwd(int32_t dtype, int64_t C, int64_t dk, int64_t dv) {
  int n = 0;
  const ll::BwdEntry* t = ll::mamba2_bwd_table(&n);
  for (int i = 0; i < n; ++i)
    if (t[i].dtype == dtype && t[i].C == C && t[i].dk == dk && t[i].dv == dv) return &t[i];
  return nullptr;
}

const ll::GdnEntry* find_gdn(int32_t dtype, int64_t C, int64_t dk, int64_t dv) {
  if (dtype != LL_BF16) return nullptr;
  int n = 0;
  const ll::GdnEntry* t = ll::gdn_table(&n);
  for (int i = 0; i < n; ++i)
    if (t[i].C == C && t[i].dk == dk && t[i].dv == dv) return &t[i];
  return nullptr;
}

ll_status check_shape(int64_t B, int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t C) {
  if (B < 1 || T < 1 || H < 1 || dk < 1 || dv < 1 || !is_pow2(C) || T % C != 0) return LL_ERR_BAD_SHAPE;
  return LL_OK;
}

}  // namespace

extern "C" {

int32_t ll_num_levels(int64_t T) { return levels_of(T); }

int32_t ll_supported(int32_t variant, int32_t dtype, int64_t C, int64_t d_k, int64_t d_v) {
  if (variant == LL_MAMBA2) return find_mamba2(dtype, C, d_k, d_v) ? 1 : 0;
  if (variant == LL_GDN) return find_gdn(dtype, C, d_k, d_v) ? 1 : 0;
  if (variant == LL_MAMBA2_BWD) return find_mamba2_bwd(dtype, C, d_k, d_v) ? 1 : 0;
  return 0;
}

size_t ll_workspace_size(int32_t variant, int32_t dtype, int64_t B, int64_t T, int64_t H, int64_t d_k, int64_t d_v,
                         int64_t C, int32_t has_lambda) {
  if (check_shape(B, T, H, d_k, d_v, C) != LL_OK) return 0;
  if (dtype != LL_F32 && dtype != LL_BF16) return 0;
  if (variant == LL_MAMBA2) {
    if (ll::mamba2_fused_supported(dtype, C, d_k, d_v, has_lambda != 0))
      return (size_t)ll::mamba2_fused_workspace(B, T, H, d_k, d_v, nullptr);
    return (size_t)ll::mamba2_workspace(B, T, H, d_k, d_v, C, elem_size(dtype), has_lambda != 0, nullptr);
  }
  if (variant == LL_GDN) return (size_t)ll::gdn_workspace(B, T, H, d_k, d_v, C, nullptr);
  if (variant == LL_MAMBA2_BWD && has_lambda)
    return (size_t)ll::mamba2_bwd_workspace(B, T, H, H, d_k, d_v, C, elem_size(dtype), nullptr);
  return 0;
}

size_t ll_mamba2_matrix_lambda_workspace_size(int32_t lambda_form, int32_t dtype, int64_t B, int64_t T, int64_t H,
                                              int64_t d_k, int64_t d_v, int64_t C) {
  if (check_shape(B, T, H, d_k, d_v, C) != LL_OK) return 0;
  if (dtype != LL_F32 && dtype != LL_BF16) return 0;
  if (lambda_form != LL_LAMBDA_DIAG && lambda_form != LL_LAMBDA_FULL) return 0;
  return (size_t)ll::mamba2_ml_workspace(B, T, H, d_k, d_v, C, elem_size(dtype), levels_of(T),
                                         lambda_form == LL_LAMBDA_FULL, nullptr);
}

size_t ll_mamba2_bwd_workspace_size(int32_t dtype, int64_t B, int64_t T, int64_t H, int64_t H_qk, int64_t d_k,
                                    int64_t d_v, int64_t C) {
  if (check_shape(B, T, H, d_k, d_v, C) != LL_OK) return 0;
  if (dtype != LL_F32 && dtype != LL_BF16) return 0;
  if (H_qk < 1 || H_qk > H || H % H_qk != 0) return 0;
  return (size_t)ll::mamba2_bwd_workspace(B, T, H, H_qk, d_k, d_v, C, elem_size(dtype), nullptr);
}

const char* ll_status_string(ll_status s) {
  switch (s) {
    case LL_OK: return "LL_OK";
    case LL_ERR_NULL_ARG: return "LL_ERR_NULL_ARG: a required pointer is NULL";
    case LL_ERR_BAD_SHAPE: return "LL_ERR_BAD_SHAPE: invalid B/T/H/d_k/d_v/C";
    case LL_ERR_UNSUPPORTED: return "LL_ERR_UNSUPPORTED: no kernel for this dtype/C/d_k/d_v";
    case LL_ERR_WORKSPACE: return "LL_ERR_WORKSPACE: workspace too small or misaligned";
    case LL_ERR_HIP: return "LL_ERR_HIP: HIP launch error";
    case LL_ERR_SCRATCH: return "LL_ERR_SCRATCH: the call needs more than the 64 MiB static device scratch";
  }
  return "unknown ll_status";
}

}  // extern "C"

namespace {
// What one log-linear Mamba-2 forward runs and the workspace it needs, from the host-side checks.
struct Mamba2Plan {
  const ll::KernelEntry* e = nullptr;
  bool fused = false;
  bool bwd_out = false;  // single-pass forward in a backward-sized workspace: leave the backward's summaries
  int L = 0;
  int64_t need = 0;
};

ll_status mamba2_plan(const void* q, const void* k, const void* v, const float* log_alpha, const float* lambda,
                      void* o, int64_t B, int64_t T, int64_t H, int64_t Hqk, int64_t d_k, int64_t d_v, int64_t C,
                      int32_t dtype, Mamba2Plan* p) {
  if (!q || !k || !v || !log_alpha || !o) return LL_ERR_NULL_ARG;
  ll_status st = check_shape(B, T, H, d_k, d_v, C);
  if (st != LL_OK) return st;
  if (Hqk < 1 || Hqk > H || H % Hqk != 0) return LL_ERR_BAD_SHAPE;
  if (dtype != LL_F32 && dtype != LL_BF16) return LL_ERR_UNSUPPORTED;
  p->e = find_mamba2(dtype, C, d_k, d_v);
  if (!p->e) return LL_ERR_UNSUPPORTED;
  p->L = levels_of(T);
  const int64_t tiles = ll::tiles_of(T, C);
  // B * H indexes the second grid dimension of the scan kernels (at most 65535)
  if (p->L > kMaxL || tiles > kMaxTiles || B * H > 65535 || tiles * 2 * H * B >= (int64_t(1) << 31))
    return LL_ERR_UNSUPPORTED;
  p->fused = ll::mamba2_fused_supported(dtype, C, d_k, d_v, lambda != nullptr);
  p->need = p->fused ? ll::mamba2_fused_workspace(B, T, H, d_k, d_v, nullptr)
                     : ll::mamba2_workspace(B, T, H, d_k, d_v, C, elem_size(dtype), lambda != nullptr, nullptr);
  return LL_OK;
}

ll_status mamba2_launch(const Mamba2Plan& p, const void* q, const void* k, const void* v, const float* log_alpha,
                        const float* lambda, void* o, int64_t B, int64_t T, int64_t H, int64_t Hqk, int64_t d_k,
                        int64_t d_v, int64_t C, void* workspace, void* stream, void* const* events) {
  ll::Mamba2Args a;
  a.q = q; a.k = k; a.v = v; a.log_alpha = log_alpha; a.lambda = lambda; a.o = o;
  a.B = B; a.T = T; a.H = H; a.dk = d_k; a.dv = d_v; a.C = C;
  a.Hqk = Hqk;
  a.L = p.L;
  a.workspace = workspace;
  a.bwd_out = p.bwd_out;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  hipEvent_t ev[ll::kMamba2Stages + 1];
  if (events)
    for (int i = 0; i <= ll::kMamba2Stages; ++i) ev[i] = static_cast<hipEvent_t>(events[i]);
  const hipError_t err =
      p.fused ? ll::launch_mamba2_fused(a, hs, events ? ev : nullptr) : p.e->launch(a, hs, events ? ev : nullptr);
  return err == hipSuccess ? LL_OK : LL_ERR_HIP;
}

ll_status mamba2_impl(const void* q, const void* k, const void* v, const float* log_alpha, const float* lambda,
                      void* o, int64_t B, int64_t T, int64_t H, int64_t Hqk, int64_t d_k, int64_t d_v, int64_t C,
                      int32_t dtype, void* workspace, size_t workspace_bytes, void* stream, void* const* events) {
  Mamba2Plan p;
  const ll_status st = mamba2_plan(q, k, v, log_alpha, lambda, o, B, T, H, Hqk, d_k, d_v, C, dtype, &p);
  if (st != LL_OK) return st;
  if (!workspace) return LL_ERR_NULL_ARG;
  if ((int64_t)workspace_bytes < p.need || (reinterpret_cast<uintptr_t>(workspace) & 255)) return LL_ERR_WORKSPACE;
  // a workspace sized for the backward: the single-pass forward also leaves the summaries that
  // ll_mamba2_bwd_after_fwd reuses
  p.bwd_out = p.fused && lambda && find_mamba2_bwd(dtype, C, d_k, d_v) &&
              (int64_t)workspace_bytes >= ll::mamba2_bwd_workspace(B, T, H, Hqk, d_k, d_v, C, elem_size(dtype), nullptr);
  return mamba2_launch(p, q, k, v, log_alpha, lambda, o, B, T, H, Hqk, d_k, d_v, C, workspace, stream, events);
}
ll_status mamba2_ml_impl(const void* q, const void* k, const void* v, const float* log_alpha, const float* Lambda,
                         int32_t form, void* o, int64_t B, int64_t T, int64_t H, int64_t d_k, int64_t d_v, int64_t C,
                         int32_t dtype, void* workspace, size_t workspace_bytes, void* stream, void* const* events) {
  if (!q || !k || !v || !log_alpha || !Lambda || !o) return LL_ERR_NULL_ARG;
  ll_status st = check_shape(B, T, H, d_k, d_v, C);
  if (st != LL_OK) return st;
  if (form != LL_LAMBDA_DIAG && form != LL_LAMBDA_FULL) return LL_ERR_BAD_SHAPE;
  if (reinterpret_cast<uintptr_t>(Lambda) & 15) return LL_ERR_BAD_SHAPE;
  if (dtype != LL_F32 && dtype != LL_BF16) return LL_ERR_UNSUPPORTED;
  const ll::KernelEntry* e = find_mamba2(dtype, C, d_k, d_v);
  if (!e) return LL_ERR_UNSUPPORTED;
  const int L = levels_of(T);
  const int64_t tiles = ll::tiles_of(T, C);
  // the tile grid and the scan grid as in the forward; one wave per (row, level) for full matrices
  if (L > kMaxL || tiles > kMaxTiles || B * H > 65535 || tiles * 2 * H * B >= (int64_t(1) << 31) ||
      B * T * H * L / 4 >= (int64_t(1) << 31))
    return LL_ERR_UNSUPPORTED;
  const int64_t need =
      ll::mamba2_ml_workspace(B, T, H, d_k, d_v, C, elem_size(dtype), L, form == LL_LAMBDA_FULL, nullptr);
  if (!workspace) return LL_ERR_NULL_ARG;
  if ((int64_t)workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)) return LL_ERR_WORKSPACE;
  ll::Mamba2Args a;
  a.q = q; a.k = k; a.v = v; a.log_alpha = log_alpha; a.lambda = nullptr; a.o = o;
  a.B = B; a.T = T; a.H = H; a.dk = d_k; a.dv = d_v; a.C = C;
  a.Hqk = H;
  a.L = L;
  a.workspace = workspace;
  a.lambda_matrix = Lambda;
  a.lambda_full = form == LL_LAMBDA_FULL;
  hipEvent_t ev[ll::kMamba2MlStages + 1];
  if (events)
    for (int i = 0; i <= ll::kMamba2MlStages; ++i) ev[i] = static_cast<hipEvent_t>(events[i]);
  const hipError_t err = e->launch_ml(a, static_cast<hipStream_t>(stream), events ? ev : nullptr);
  return err == hipSuccess ? LL_OK : LL_ERR_HIP;
}
ll_status mamba2_bwd_impl(const void* q, const void* k, const void* v, const float* log_alpha, const float* lambda,
                          const void* d_o, void* dq, void* dk, void* dv, float* dlog_alpha, float* dlambda, int64_t B,
                          int64_t T, int64_t H, int64_t Hqk, int64_t d_k, int64_t d_v, int64_t C, int32_t dtype,
                          void* workspace, size_t workspace_bytes, void* stream, void* const* events, bool reuse) {
  if (!q || !k || !v || !log_alpha || !lambda || !d_o || !dq || !dk || !dv || !dlog_alpha || !dlambda)
    return LL_ERR_NULL_ARG;
  ll_status st = check_shape(B, T, H, d_k, d_v, C);
  if (st != LL_OK) return st;
  if (Hqk < 1 || Hqk > H || H % Hqk != 0) return LL_ERR_BAD_SHAPE;
  if (dtype != LL_F32 && dtype != LL_BF16) return LL_ERR_UNSUPPORTED;
  const ll::BwdEntry* e = find_mamba2_bwd(dtype, C, d_k, d_v);
  if (!e) return LL_ERR_UNSUPPORTED;
  const int L = levels_of(T);
  const int64_t tiles = ll::tiles_of(T, C);
  // B * H indexes the second / third grid dimension of the scan, reduce and gate kernels; the
  // group sums launch one thread per output element
  if (L > kMaxL || tiles > kMaxTiles || B * H > 65535 || tiles * H * B >= (int64_t(1) << 31) ||
      B * T * Hqk * d_k / 256 >= (int64_t(1) << 31))
    return LL_ERR_UNSUPPORTED;
  const int64_t need = ll::mamba2_bwd_workspace(B, T, H, Hqk, d_k, d_v, C, elem_size(dtype), nullptr);
  if (!workspace) return LL_ERR_NULL_ARG;
  if ((int64_t)workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)) return LL_ERR_WORKSPACE;
  ll::Mamba2BwdArgs a;
  a.q = q; a.k = k; a.v = v; a.dout = d_o; a.log_alpha = log_alpha; a.lambda = lambda;
  a.dq = dq; a.dk = dk; a.dv = dv; a.dlog_alpha = dlog_alpha; a.dlambda = dlambda;
  a.B = B; a.T = T; a.H = H; a.C = C;
  a.Hqk = Hqk;
  a.L = L;
  a.workspace = workspace;
  a.reuse_summaries = reuse;
  a.fused_fwd = ll::mamba2_fused_supported(dtype, C, d_k, d_v, true);
  hipEvent_t ev[ll::kMamba2BwdStages + 1];
  if (events)
    for (int i = 0; i <= ll::kMamba2BwdStages; ++i) ev[i] = static_cast<hipEvent_t>(events[i]);
  const hipError_t err = e->launch(a, static_cast<hipStream_t>(stream), events ? ev : nullptr);
  return err == hipSuccess ? LL_OK : LL_ERR_HIP;
}
ll_status gdn_impl(const void* q, const void* k, const void* v, const float* log_alpha, const float* beta,
                   const float* lambda, void* o, int64_t B, int64_t T, int64_t H, int64_t d_k, int64_t d_v, int64_t C,
                   int32_t dtype, void* workspace, size_t workspace_bytes, void* stream, void* const* events) {
  if (!q || !k || !v || !log_alpha || !beta || !o) return LL_ERR_NULL_ARG;
  ll_status st = check_shape(B, T, H, d_k, d_v, C);
  if (st != LL_OK) return st;
  const ll::GdnEntry* e = find_gdn(dtype, C, d_k, d_v);
  if (!e) return LL_ERR_UNSUPPORTED;
  const int64_t N = T / C;
  const int J = N <= 1 ? 0 : bitlen64(uint64_t(N - 1));
  const int L = levels_of(T);
  if (J > ll::kGdnMaxLevels || L > kMaxL || H > 65535 || B > 65535 || B * H * N >= (int64_t(1) << 31))
    return LL_ERR_UNSUPPORTED;
  const int64_t need = ll::gdn_workspace(B, T, H, d_k, d_v, C, nullptr);
  if (!workspace) return LL_ERR_NULL_ARG;
  if ((int64_t)workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255)) return LL_ERR_WORKSPACE;
  ll::GdnArgs a;
  a.q = q; a.k = k; a.v = v; a.log_alpha = log_alpha; a.beta = beta; a.lambda = lambda; a.o = o;
  a.B = B; a.T = T; a.H = H; a.dk = d_k; a.dv = d_v; a.C = C;
  a.L = L;
  a.workspace = workspace;
  hipEvent_t ev[ll::kGdnStages + 1];
  if (events)
    for (int i = 0; i <= ll::kGdnStages; ++i) ev[i] = static_cast<hipEvent_t>(events[i]);
  const hipError_t err = e->launch(a, static_cast<hipStream_t>(stream), events ? ev : nullptr);
  return err == hipSuccess ? LL_OK : LL_ERR_HIP;
}
}  // namespace

extern "C" {

ll_status ll_mamba2_fwd(const void* q, const void* k, const void* v, const float* log_alpha, const float* lambda,
                        void* o, int64_t B, int64_t T, int64_t H, int64_t d_k, int64_t d_v, int64_t C, int32_t dtype,
                        void* workspace, size_t workspace_bytes, void* stream) {
  return mamba2_impl(q, k, v, log_alpha, lambda, o, B, T, H, H, d_k, d_v, C, dtype, workspace, workspace_bytes, stream,
                     nullptr);
}

ll_status ll_mamba2_fwd_grouped(const void* q, const void* k, const void* v, const float* log_alpha,
                                const float* lambda, void* o, int64_t B, int64_t T, int64_t H, int64_t H_qk,
                                int64_t d_k, int64_t d_v, int64_t C, int32_t dtype, void* workspace,
                                size_t workspace_bytes, void* stream) {
  return mamba2_impl(q, k, v, log_alpha, lambda, o, B, T, H, H_qk, d_k, d_v, C, dtype, workspace, workspace_bytes,
                     stream, nullptr);
}

ll_status ll_mamba2_fwd_staged(const void* q, const void* k, const void* v, const float* log_alpha,
                               const float* lambda, void* o, int64_t B, int64_t T, int64_t H, int64_t H_qk,
                               int64_t d_k, int64_t d_v, int64_t C, int32_t dtype, void* workspace,
                               size_t workspace_bytes, void* stream, void* const* events) {
  if (!events) return LL_ERR_NULL_ARG;
  for (int i = 0; i <= ll::kMamba2Stages; ++i)
    if (!events[i]) return LL_ERR_NULL_ARG;
  return mamba2_impl(q, k, v, log_alpha, lambda, o, B, T, H, H_qk, d_k, d_v, C, dtype, workspace, workspace_bytes,
                     stream, events);
}

ll_status ll_mamba2_fwd_matrix_lambda(const void* q, const void* k, const void* v, const float* log_alpha,
                                      const float* Lambda, int32_t lambda_form, void* o, int64_t B, int64_t T,
                                      int64_t H, int64_t d_k, int64_t d_v, int64_t C, int32_t dtype, void* workspace,
                                      size_t workspace_bytes, void* stream) {
  return mamba2_ml_impl(q, k, v, log_alpha, Lambda, lambda_form, o, B, T, H, d_k, d_v, C, dtype, workspace,
                        workspace_bytes, stream, nullptr);
}

ll_status ll_mamba2_fwd_matrix_lambda_staged(const void* q, const void* k, const void* v, const float* log_alpha,
                                             const float* Lambda, int32_t lambda_form, void* o, int64_t B, int64_t T,
                                             int64_t H, int64_t d_k, int64_t d_v, int64_t C, int32_t dtype,
                                             void* workspace, size_t workspace_bytes, void* stream,
                                             void* const* events) {
  if (!events) return LL_ERR_NULL_ARG;
  for (int i = 0; i <= ll::kMamba2MlStages; ++i)
    if (!events[i]) return LL_ERR_NULL_ARG;
  return mamba2_ml_impl(q, k, v, log_alpha, Lambda, lambda_form, o, B, T, H, d_k, d_v, C, dtype, workspace,
                        workspace_bytes, stream, events);
}

ll_status ll_mamba2_bwd(const void* q, const void* k, const void* v, const float* log_alpha, const float* lambda,
                        const void* d_o, void* dq, void* dk, void* dv, float* dlog_alpha, float* dlambda, int64_t B,
                        int64_t T, int64_t H, int64_t d_k, int64_t d_v, int64_t C, int32_t dtype, void* workspace,
                        size_t workspace_bytes, void* stream) {
  return mamba2_bwd_impl(q, k, v, log_alpha, lambda, d_o, dq, dk, dv, dlog_alpha, dlambda, B, T, H, H, d_k, d_v, C,
                         dtype, workspace, workspace_bytes, stream, nullptr, false);
}

ll_status ll_mamba2_bwd_grouped(const void* q, const void* k, const void* v, const float* log_alpha,
                                const float* lambda, const void* d_o, void* dq, void* dk, void* dv, float* dlog_alpha,
                                float* dlambda, int64_t B, int64_t T, int64_t H, int64_t H_qk, int64_t d_k, int64_t d_v,
                                int64_t C, int32_t dtype, void* workspace, size_t workspace_bytes, void* stream) {
  return mamba2_bwd_impl(q, k, v, log_alpha, lambda, d_o, dq, dk, dv, dlog_alpha, dlambda, B, T, H, H_qk, d_k, d_v, C,
                         dtype, workspace, workspace_bytes, stream, nullptr, false);
}

ll_status ll_mamba2_bwd_after_fwd(const void* q, const void* k, const void* v, const float* log_alpha,
                                  const float* lambda, const void* d_o, void* dq, void* dk, void* dv, float* dlog_alpha,
                                  float* dlambda, int64_t B, int64_t T, int64_t H, int64_t H_qk, int64_t d_k,
                                  int64_t d_v, int64_t C, int32_t dtype, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  return mamba2_bwd_impl(q, k, v, log_alpha, lambda, d_o, dq, dk, dv, dlog_alpha, dlambda, B, T, H, H_qk, d_k, d_v, C,
                         dtype, workspace, workspace_bytes, stream, nullptr, true);
}

ll_status ll_mamba2_bwd_staged(const void* q, const void* k, const void* v, const float* log_alpha,
                               const float* lambda, const void* d_o, void* dq, void* dk, void* dv, float* dlog_alpha,
                               float* dlambda, int64_t B, int64_t T, int64_t H, int64_t H_qk, int64_t d_k, int64_t d_v,
                               int64_t C, int32_t dtype, void* workspace, size_t workspace_bytes, void* stream,
                               void* const* events) {
  if (!events) return LL_ERR_NULL_ARG;
  for (int i = 0; i <= ll::kMamba2BwdStages; ++i)
    if (!events[i]) return LL_ERR_NULL_ARG;
  return mamba2_bwd_impl(q, k, v, log_alpha, lambda, d_o, dq, dk, dv, dlog_alpha, dlambda, B, T, H, H_qk, d_k, d_v, C,
                         dtype, workspace, workspace_bytes, stream, events, false);
}

ll_status ll_gdn_fwd(const void* q, const void* k, const void* v, const float* log_alpha, const float* beta,
                     const float* lambda, void* o, int64_t B, int64_t T, int64_t H, int64_t d_k, int64_t d_v, int64_t C,
                     int32_t dtype, void* workspace, size_t workspace_bytes, void* stream) {
  return gdn_impl(q, k, v, log_alpha, beta, lambda, o, B, T, H, d_k, d_v, C, dtype, workspace, workspace_bytes, stream,
                  nullptr);
}

ll_status ll_gdn_fwd_staged(const void* q, const void* k, const void* v, const float* log_alpha, const float* beta,
                            const float* lambda, void* o, int64_t B, int64_t T, int64_t H, int64_t d_k, int64_t d_v,
                            int64_t C, int32_t dtype, void* workspace, size_t workspace_bytes, void* stream,
                            void* const* events) {
  if (!events) return LL_ERR_NULL_ARG;
  for (int i = 0; i <= ll::kGdnStages; ++i)
    if (!events[i]) return LL_ERR_NULL_ARG;
  return gdn_impl(q, k, v, log_alpha, beta, lambda, o, B, T, H, d_k, d_v, C, dtype, workspace, workspace_bytes, stream,
                  events);
}

}  // extern "C"

// ---- forward without allocation ----------------------------------------------------------------
// The workspace of ll_mamba2_fwd_noalloc: each GPU the library runs on holds one copy of this
// array until the process ends.  In host code the name stands for a host-side shadow, not a device
// address: host code only ever uses the address scratch_ptr() looked up for the device.
static __device__ __align__(256) unsigned char scratch[LL_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];  // device address of `scratch`, per device
std::mutex g_scratch_mu;                    // serialises the one look-up per device

// The device address of `scratch` on the device that `stream` belongs to (the current device for
// the NULL stream), looked up on that device's first call with the device current.
ll_status scratch_ptr(void* stream, void** out) {
  int dev = -1;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (hs) {
    hipDevice_t d = -1;
    if (hipStreamGetDevice(hs, &d) != hipSuccess) return LL_ERR_HIP;
    dev = d;
  } else if (hipGetDevice(&dev) != hipSuccess) {
    return LL_ERR_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) return LL_ERR_UNSUPPORTED;
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (!p) {
      int cur = -1;
      if (hipGetDevice(&cur) != hipSuccess) return LL_ERR_HIP;
      if (cur != dev && hipSetDevice(dev) != hipSuccess) return LL_ERR_HIP;
      const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (cur != dev) (void)hipSetDevice(cur);
      if (e != hipSuccess || !p) return LL_ERR_HIP;
      g_scratch[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return LL_OK;
}
}  // namespace

extern "C" {

ll_status ll_mamba2_fwd_noalloc(const void* q, const void* k, const void* v, const float* log_alpha,
                                const float* lambda, void* o, int64_t B, int64_t T, int64_t H, int64_t d_k,
                                int64_t d_v, int64_t C, int32_t dtype, void* stream) {
  Mamba2Plan p;
  ll_status st = mamba2_plan(q, k, v, log_alpha, lambda, o, B, T, H, H, d_k, d_v, C, dtype, &p);
  if (st != LL_OK) return st;
  if (p.need > (int64_t)LL_NOALLOC_SCRATCH_BYTES) return LL_ERR_SCRATCH;
  void* ws = nullptr;
  st = scratch_ptr(stream, &ws);
  if (st != LL_OK) return st;
  return mamba2_launch(p, q, k, v, log_alpha, lambda, o, B, T, H, H, d_k, d_v, C, ws, stream, nullptr);
}

ll_status ll_debug_level_map(int64_t T, int64_t C, int8_t* out, void* stream) {
  if (!out) return LL_ERR_NULL_ARG;
  if (T < 1 || !is_pow2(C) || T % C != 0) return LL_ERR_BAD_SHAPE;
  if (T > 16384) return LL_ERR_UNSUPPORTED;
  hipError_t err = ll::launch_debug_level_map(T, C, out, static_cast<hipStream_t>(stream));
  return err == hipSuccess ? LL_OK : LL_ERR_HIP;
}

}  // extern "C"
