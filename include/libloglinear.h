/*
 * libloglinear — chunkwise-parallel forward pass of log-linear attention on AMD MI355X (gfx950).
 *
 * Method: Guo et al., "Log-Linear Attention".  The library computes, per batch b and head h,
 *
 *     O = (Q K^T  (.)  M^S  (.)  M^H) V                        log-linear Mamba-2      (Sec. 3.4)
 *     O = (A  (.)  M^S  (.)  M^H) V,
 *         A = (Q K^T (.) L)(I + diag(beta)(K K^T (.) (L - I)))^{-1} diag(beta)
 *                                                              log-linear Gated DeltaNet (Sec. 3.4)
 *
 * where M^S[t,s] = prod_{k=s+1..t} alpha_k is the gated (semiseparable) decay mask (Eq. 2),
 * M^H[t,s] = lambda_t^(l(t,s)) is the Fenwick-tree hierarchical mask (Eq. 4) with l(t,s) the
 * Fenwick level of position s seen from t (Sec. 3.1), and L is the lower-triangular ones matrix.
 * It uses the chunkwise algorithm of Sec. 3.3 (Eq. 5): a dense C x C intra-chunk stage and
 * O(log(T/C)) inter-chunk levels.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Layout.   All tensors are dense, row-major, in device memory:
 *             q, k         [B, T, H, d_k]
 *             v, o         [B, T, H, d_v]
 *             log_alpha    [B, T, H]         (float32, log of alpha_t; the caller keeps it <= 0)
 *             beta         [B, T, H]         (float32, GDN only)
 *             lambda       [B, T, H, L]      (float32, L = ll_num_levels(T); the caller keeps it >= 0)
 *           q, k, v and o share one storage dtype (ll_dtype); gates, beta and lambda are float32.
 *           NaN or Inf in any input propagates to o; values are not checked.
 * Shapes.   B, H >= 1; T >= 1 and T % C == 0; C a power of two; (dtype, C, d_k, d_v) must be one of
 *           the compiled kernel shapes (ll_supported).  Size limits (LL_ERR_UNSUPPORTED beyond them):
 *           L <= 24 levels; for log-linear Mamba-2 at most 8192 tiles of max(2C, 64) tokens per
 *           sequence and B * H <= 65535.
 * Ownership. Every pointer is caller-owned device memory.  The library allocates nothing (the one
 *           static device array of ll_mamba2_fwd_noalloc aside), keeps no pointer after the call
 *           returns, and enqueues all work on `stream` (a hipStream_t passed as void*, NULL = the
 *           default stream).  Calls return before the work finishes: the caller keeps all buffers
 *           alive and unmodified until the stream reaches this point.
 * Workspace. Device scratch of at least ll_workspace_size(...) bytes, 256-byte aligned, owned by the
 *           caller; its contents on entry are irrelevant.  Calls sharing a workspace must be ordered.
 * Errors.   Argument checks run on the host before any launch; on error nothing is enqueued.
 *           A failed launch returns LL_ERR_HIP.  No exceptions cross the ABI.  Thread-safe: the
 *           only mutable global state is ll_mamba2_fwd_noalloc's per-device scratch (see there).
 */
#ifndef LIBLOGLINEAR_H
#define LIBLOGLINEAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LL_OK = 0,
  LL_ERR_NULL_ARG = 1,     /* a required pointer is NULL                                        */
  LL_ERR_BAD_SHAPE = 2,    /* B, T or H < 1, T % C != 0, C not a power of two, or d_k/d_v < 1   */
  LL_ERR_UNSUPPORTED = 3,  /* no compiled kernel for (dtype, C, d_k, d_v), an unknown dtype, or
                              sizes beyond the limits stated under Shapes                        */
  LL_ERR_WORKSPACE = 4,    /* workspace smaller than ll_workspace_size(...) or misaligned       */
  LL_ERR_HIP = 5,          /* the HIP runtime reported an error when launching                   */
  LL_ERR_SCRATCH = 6       /* ll_mamba2_fwd_noalloc: the call needs more device scratch than
                              LL_NOALLOC_SCRATCH_BYTES                                          */
} ll_status;

/* Bytes of the static device scratch ll_mamba2_fwd_noalloc works in (one copy per GPU). */
#define LL_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

typedef enum { LL_F32 = 0, LL_BF16 = 1 } ll_dtype;

typedef enum { LL_MAMBA2 = 0, LL_GDN = 1, LL_MAMBA2_BWD = 2 } ll_variant;  /* LL_MAMBA2_BWD: the backward call */

/* Number of Fenwick levels L for a sequence of length T (Sec. 3.1): one more than the largest
 * level l(t,s) over all 0 <= s <= t < T, i.e. ceil(log2 T) + 1 for T >= 2 and 1 for T = 1.
 * Returns -1 for T < 1.  Pure host function. */
int32_t ll_num_levels(int64_t T);

/* 1 if a kernel is compiled for this (variant, dtype, C, d_k, d_v), else 0.  Pure host function. */
int32_t ll_supported(int32_t variant, int32_t dtype, int64_t C, int64_t d_k, int64_t d_v);

/* Bytes of workspace the forward call needs for these arguments; `has_lambda` = 0 sizes the
 * lambda == NULL path.  With variant LL_MAMBA2_BWD: bytes for ll_mamba2_bwd (has_lambda must be
 * 1).  Returns 0 if the arguments are invalid.  Pure host function. */
size_t ll_workspace_size(int32_t variant, int32_t dtype, int64_t B, int64_t T, int64_t H,
                         int64_t d_k, int64_t d_v, int64_t C, int32_t has_lambda);

/* Log-linear Mamba-2 forward, O = (Q K^T (.) M^S (.) M^H) V (Sec. 3.4; chunkwise algorithm
 * Sec. 3.3, Eq. 5).  lambda == NULL sets all level weights to 1, which is exactly Mamba-2 /
 * gated linear attention (Eq. 2): bf16 with C = 64 runs the same single-pass kernels with unit
 * weights, the other shapes one running state between chunks.  Arguments as in the conventions
 * above; o is written in full. */
ll_status ll_mamba2_fwd(const void* q, const void* k, const void* v, const float* log_alpha,
                        const float* lambda, void* o, int64_t B, int64_t T, int64_t H,
                        int64_t d_k, int64_t d_v, int64_t C, int32_t dtype,
                        void* workspace, size_t workspace_bytes, void* stream);

/* ll_mamba2_fwd for callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops, harnesses that forbid hipMalloc): the same kernels and the same result as
 * ll_mamba2_fwd, with the workspace taken from a static device array of LL_NOALLOC_SCRATCH_BYTES
 * (64 MiB) instead of an argument.  The caller still owns q, k, v, log_alpha, lambda and o.
 * Each GPU holds its own copy of the array from the first call on that GPU (whose device address
 * is looked up then, with the stream's device current) until the process ends.  Nothing is
 * allocated, on the device or the host, by this call.
 * Limits.   Arguments whose ll_workspace_size(LL_MAMBA2, ...) exceeds LL_NOALLOC_SCRATCH_BYTES
 *           return LL_ERR_SCRATCH before anything is enqueued; e.g. bf16 with C = 64 and
 *           d_k = d_v = 128 needs about 256 bytes per token and head (B * T * H up to about 2^18).
 * Sharing.  Every call on one GPU works in that GPU's one array and leaves its contents behind
 *           (the kernels clear what must start at zero): calls on one GPU must be ordered (one
 *           stream, or streams joined by events); calls that overlap on one GPU race and give
 *           wrong results.  Other errors as ll_mamba2_fwd. */
ll_status ll_mamba2_fwd_noalloc(const void* q, const void* k, const void* v, const float* log_alpha,
                                const float* lambda, void* o, int64_t B, int64_t T, int64_t H,
                                int64_t d_k, int64_t d_v, int64_t C, int32_t dtype, void* stream);

/* Log-linear Mamba-2 forward with query/key heads shared by groups of heads: q and k are
 * [B, T, H_qk, d_k] and head h (of H) uses query/key head h / (H / H_qk); v, o, log_alpha and
 * lambda keep H heads.  H_qk = 1 is the multi-value form of Mamba-2 (one B/C projection for
 * every head), 1 < H_qk < H the grouped form; H_qk = H is ll_mamba2_fwd.  The result equals
 * ll_mamba2_fwd on q and k repeated across each group.  H_qk < 1, H_qk > H or H % H_qk != 0
 * returns LL_ERR_BAD_SHAPE; otherwise as ll_mamba2_fwd (same workspace size for the same H). */
ll_status ll_mamba2_fwd_grouped(const void* q, const void* k, const void* v, const float* log_alpha,
                                const float* lambda, void* o, int64_t B, int64_t T, int64_t H,
                                int64_t H_qk, int64_t d_k, int64_t d_v, int64_t C, int32_t dtype,
                                void* workspace, size_t workspace_bytes, void* stream);

/* Same computation as ll_mamba2_fwd_grouped (ll_mamba2_fwd for H_qk = H), for measurement:
 * also records the caller's HIP events
 * (hipEvent_t handles passed as void*) on `stream`, events[i] right before kernel stage i and
 * events[3] after the last stage, so that the caller can read each stage's duration with
 * hipEventElapsedTime once the stream has passed them.  Stages of the single-pass path (bf16,
 * C = 64): 0 tile totals of the log-gates, 1 aligned block sums of those totals, 2 the tile
 * kernel (states, Fenwick nodes, intra-tile and inter-tile terms).  Stages of the three-kernel
 * path: 0 tile states and the summaries of the lowest three tile levels, 1 scan (the block tree
 * of summaries above them; with lambda == NULL the running state of every tile), 2 tile outputs
 * (intra-tile and inter-tile terms).  Asynchronous like ll_mamba2_fwd.  events
 * == NULL or any events[i] == NULL returns LL_ERR_NULL_ARG; the events stay owned by the caller. */
ll_status ll_mamba2_fwd_staged(const void* q, const void* k, const void* v, const float* log_alpha,
                               const float* lambda, void* o, int64_t B, int64_t T, int64_t H,
                               int64_t H_qk, int64_t d_k, int64_t d_v, int64_t C, int32_t dtype,
                               void* workspace, size_t workspace_bytes, void* stream,
                               void* const* events);

/* ---- Matrix-valued level weights (the 4D-tensor view of App. A) ------------------------------
 *
 * App. A writes a pair's score as q_t M[t,s] k_s^T with a d_k x d_k matrix per pair; log-linear
 * Mamba-2 with matrix-valued weights takes M[t,s] = Lambda_t^(l(t,s)) prod_{r=s+1..t} alpha_r, so
 *     O_t = sum_{s <= t} prod(alpha) (q_t Lambda_t^(l(t,s)) . k_s) v_s
 * (q_t a row vector).  lambda_t^(l) I gives ll_mamba2_fwd.  Computed as ll_mamba2_fwd is, with the
 * level queries q_t Lambda_t^(l), rounded once to the storage dtype, in place of q: each score tile
 * uses the queries of its level.  Full matrices: the level queries are formed first, into the
 * workspace; diagonal ones: the tile kernel scales its query fragments as it needs them.
 *
 * Lambda is float32, 16-byte aligned, in one of two layouts (lambda_form):
 *   LL_LAMBDA_DIAG  [B, T, H, L, d_k]        Lambda_t^(l) = diag(Lambda[b, t, h, l, :]);
 *   LL_LAMBDA_FULL  [B, T, H, L, d_k, d_k]   (Lambda_t^(l))_{a c} = Lambda[b, t, h, l, a, c].
 * L = ll_num_levels(T).  Every (dtype, C, d_k, d_v) of ll_mamba2_fwd is supported; the query and
 * key heads are not shared (H_qk = H).  The workspace is
 * ll_mamba2_matrix_lambda_workspace_size(lambda_form, ...) bytes: the forward's summaries (the
 * size ll_workspace_size gives with lambda), plus B * T * H * L * d_k level queries for full
 * matrices; 0 for invalid arguments.  An unknown lambda_form or a misaligned Lambda gives
 * LL_ERR_BAD_SHAPE; B * T * H * L >= 2^33 gives LL_ERR_UNSUPPORTED; otherwise as ll_mamba2_fwd. */
typedef enum { LL_LAMBDA_DIAG = 0, LL_LAMBDA_FULL = 1 } ll_lambda_form;

size_t ll_mamba2_matrix_lambda_workspace_size(int32_t lambda_form, int32_t dtype, int64_t B,
                                              int64_t T, int64_t H, int64_t d_k, int64_t d_v,
                                              int64_t C);

ll_status ll_mamba2_fwd_matrix_lambda(const void* q, const void* k, const void* v,
                                      const float* log_alpha, const float* Lambda,
                                      int32_t lambda_form, void* o, int64_t B, int64_t T, int64_t H,
                                      int64_t d_k, int64_t d_v, int64_t C, int32_t dtype,
                                      void* workspace, size_t workspace_bytes, void* stream);

/* As ll_mamba2_fwd_matrix_lambda, recording five caller-owned HIP events on `stream`: before the
 * level queries (no kernel for diagonal weights), the tile states, the scan and the tile outputs,
 * and after the tile outputs.
 * events == NULL or any events[i] == NULL gives LL_ERR_NULL_ARG. */
ll_status ll_mamba2_fwd_matrix_lambda_staged(const void* q, const void* k, const void* v,
                                             const float* log_alpha, const float* Lambda,
                                             int32_t lambda_form, void* o, int64_t B, int64_t T,
                                             int64_t H, int64_t d_k, int64_t d_v, int64_t C,
                                             int32_t dtype, void* workspace, size_t workspace_bytes,
                                             void* stream, void* const* events);

/* ---- Backward pass of log-linear Mamba-2 -----------------------------------------------------
 *
 * Gradients of the scalar sum(O (.) dO) for O = (Q K^T (.) M^S (.) M^H) V (Sec. 3.4), with respect
 * to every input.  Per (b, h), with w(t, s) = lambda_t^(l(t,s)) exp(cum_t - cum_s) (s <= t),
 * cum the running sum of log_alpha, P = Q K^T and G = dO V^T:
 *   dq = (w (.) G) K,   dk = (w (.) G)^T Q,   dv = (w (.) P)^T dO,
 *   dlambda_t^(l) = sum over s at level l of exp(cum_t - cum_s) P[t,s] G[t,s]  (0 for levels no
 *                   pair of row t reaches),
 *   dlog_alpha_tau = sum over t >= tau of (q_t . dq_t - k_t . dk_t).
 * Computed chunkwise like the forward (Sec. 3.3): the forward's level summaries for the query
 * side, and per-level summaries of later tokens (lambda-weighted, since lambda belongs to the
 * query) for the key side.  The forward output is not needed.
 *
 * d_o, dq, dk, dv have the layout and storage dtype of v, q, k, v; dlog_alpha [B, T, H] and
 * dlambda [B, T, H, L] are float32.  Every output is written in full (caller-owned device
 * memory, not read).  lambda is required (pass ones for Mamba-2): NULL gives LL_ERR_NULL_ARG.
 * Shapes, dtypes and compiled (C, d_k, d_v) as for ll_mamba2_fwd; the workspace is
 * ll_workspace_size(LL_MAMBA2_BWD, ...) bytes.  Asynchronous on `stream`. */
ll_status ll_mamba2_bwd(const void* q, const void* k, const void* v, const float* log_alpha,
                        const float* lambda, const void* d_o, void* dq, void* dk, void* dv,
                        float* dlog_alpha, float* dlambda, int64_t B, int64_t T, int64_t H,
                        int64_t d_k, int64_t d_v, int64_t C, int32_t dtype,
                        void* workspace, size_t workspace_bytes, void* stream);

/* ll_mamba2_bwd reusing the forward's level summaries instead of recomputing them: for a backward
 * that follows ll_mamba2_fwd_grouped (ll_mamba2_fwd for H_qk = H) with non-NULL lambda on the same
 * inputs, run with this same workspace (ll_mamba2_bwd_workspace_size(...) bytes: the forward uses
 * its leading part and leaves its summaries there), on the same stream or ordered after it.  The
 * summaries depend on the shapes, k, v and log_alpha only; the forward records those (shapes and
 * pointers) beside them, and the backward compares that record on the device with its own
 * arguments: on a mismatch (another forward, another workspace user in between, other inputs) every
 * gradient is written as NaN instead.  Inputs changed in place at the same addresses are not
 * detected.  For the shapes whose forward is the single-pass kernel (bf16, C = 64), a forward
 * given this workspace also stores every Fenwick node it publishes in the backward's order, with
 * the tiles' cumulative gates (any other forward in the buffer, lambda == NULL or with a smaller
 * workspace_bytes, clears the record); the gradients then differ from ll_mamba2_bwd's by the
 * rounding of those bf16 summaries.  Arguments and checks as ll_mamba2_bwd_grouped. */
ll_status ll_mamba2_bwd_after_fwd(const void* q, const void* k, const void* v, const float* log_alpha,
                                  const float* lambda, const void* d_o, void* dq, void* dk, void* dv,
                                  float* dlog_alpha, float* dlambda, int64_t B, int64_t T, int64_t H,
                                  int64_t H_qk, int64_t d_k, int64_t d_v, int64_t C, int32_t dtype,
                                  void* workspace, size_t workspace_bytes, void* stream);

/* Backward of ll_mamba2_fwd_grouped: q, k, dq and dk are [B, T, H_qk, d_k]; head h (of H) reads
 * query/key head h / (H / H_qk), so dq and dk of a shared head sum the gradients of its group of
 * heads.  H_qk < 1, H_qk > H or H % H_qk != 0 gives LL_ERR_BAD_SHAPE; the workspace is
 * ll_mamba2_bwd_workspace_size(dtype, B, T, H, H_qk, d_k, d_v, C) bytes (H_qk < H adds per-head
 * dq and dk scratch); otherwise as ll_mamba2_bwd, which is the case H_qk = H. */
ll_status ll_mamba2_bwd_grouped(const void* q, const void* k, const void* v, const float* log_alpha,
                                const float* lambda, const void* d_o, void* dq, void* dk, void* dv,
                                float* dlog_alpha, float* dlambda, int64_t B, int64_t T, int64_t H,
                                int64_t H_qk, int64_t d_k, int64_t d_v, int64_t C, int32_t dtype,
                                void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes of the backward calls for H_qk query/key heads (0 if an argument is invalid);
 * equals ll_workspace_size(LL_MAMBA2_BWD, ..., 1) for H_qk = H.  Pure host function. */
size_t ll_mamba2_bwd_workspace_size(int32_t dtype, int64_t B, int64_t T, int64_t H, int64_t H_qk,
                                    int64_t d_k, int64_t d_v, int64_t C);

/* Same computation as ll_mamba2_bwd_grouped, for measurement, recording the caller's HIP events on
 * `stream`: events[i] right before stage i and events[4] after the last.  Stages: 0 the forward's
 * level summaries, 1 the key-side level summaries, 2 dq and dlambda, 3 dk, dv and dlog_alpha.
 * events == NULL or any events[i] == NULL returns LL_ERR_NULL_ARG. */
ll_status ll_mamba2_bwd_staged(const void* q, const void* k, const void* v, const float* log_alpha,
                               const float* lambda, const void* d_o, void* dq, void* dk, void* dv,
                               float* dlog_alpha, float* dlambda, int64_t B, int64_t T, int64_t H,
                               int64_t H_qk, int64_t d_k, int64_t d_v, int64_t C, int32_t dtype,
                               void* workspace, size_t workspace_bytes, void* stream,
                               void* const* events);

/* ---- Decoding (one token at a time, Sec. 3.2) -------------------------------------------------
 *
 * Log-linear Mamba-2 keeps, per (b, h), one state per Fenwick level: O(log t) states of d_v x d_k.
 * Token t (0-based) updates them as Sec. 3.2 describes, gated: for t >= 1, with p = lssb(t), level
 * p+1 takes the sum of levels 0..p, levels 1..p are emptied, the others carry over, every carried
 * or merged level is multiplied by alpha_t, and level 0 becomes v_t k_t^T; the output is
 * o_t = sum_l lambda_t^(l) S_t^(l) q_t (Eq. 3).  Feeding tokens 0..T-1 in order gives the rows of
 * ll_mamba2_fwd on the same sequence.
 *
 * The state lives in one caller-owned device buffer of ll_decode_state_bytes(B, H, d_k, d_v, L)
 * bytes, 256-byte aligned, whose layout is private to the library; L levels hold tokens
 * t < 2^(L-1) (L = ll_num_levels(T) for a sequence of T tokens, at most 32).  Per-token tensors
 * are q, k [B, H, d_k], v, o [B, H, d_v] in the storage dtype, log_alpha [B, H] and lambda
 * [B, H, L] float32 (lambda == NULL: all level weights 1, i.e. Mamba-2 decoding).  Supported
 * (dtype, d_k, d_v): fp32 (16, 16), (64, 64); bf16 (64, 64), (128, 64), (128, 128).  Steps on one
 * state must be enqueued in token order on one stream (each step reads what the previous one
 * wrote); the state is read and written in place. */

/* Bytes of decode state for these sizes; 0 if an argument is < 1.  Pure host function. */
size_t ll_decode_state_bytes(int64_t B, int64_t H, int64_t d_k, int64_t d_v, int32_t L);

/* Resets a decode state to the empty sequence (enqueued on `stream`). */
ll_status ll_mamba2_decode_init(void* state, size_t state_bytes, int64_t B, int64_t H, int64_t d_k,
                                int64_t d_v, int32_t L, int32_t dtype, void* stream);

/* Feeds token t to every (b, h) and writes its output o.  t must be the number of tokens fed
 * since the last ll_mamba2_decode_init and below 2^(L-1) (else LL_ERR_BAD_SHAPE); a state
 * buffer too small or misaligned gives LL_ERR_WORKSPACE; an uncompiled (dtype, d_k, d_v),
 * L > 32 or B*H > 65535 gives LL_ERR_UNSUPPORTED. */
ll_status ll_mamba2_decode_step(const void* q, const void* k, const void* v, const float* log_alpha,
                                const float* lambda, void* o, void* state, size_t state_bytes,
                                int64_t t, int64_t B, int64_t H, int64_t d_k, int64_t d_v,
                                int32_t L, int32_t dtype, void* stream);

/* Log-linear Gated DeltaNet decoding with the same state buffer (ll_decode_state_bytes) and
 * conventions.  Token t applies the gated delta-rule transition alpha_t (I - beta_t k_t k_t^T) to
 * every carried and merged level (Sec. 3.2 merges; every nonempty level is rewritten each step),
 * then beta_t v_t k_t^T enters level 0; o_t = sum_l lambda_t^(l) S_t^(l) q_t.  beta [B, H] is
 * float32 and required; lambda == NULL gives Gated DeltaNet decoding.  Feeding tokens 0..T-1 gives
 * the rows of the log-linear Gated DeltaNet forward.  Same shapes, checks and statuses as the
 * Mamba-2 calls (a state is used by one variant between initialisations). */
ll_status ll_gdn_decode_init(void* state, size_t state_bytes, int64_t B, int64_t H, int64_t d_k,
                             int64_t d_v, int32_t L, int32_t dtype, void* stream);
ll_status ll_gdn_decode_step(const void* q, const void* k, const void* v, const float* log_alpha,
                             const float* beta, const float* lambda, void* o, void* state,
                             size_t state_bytes, int64_t t, int64_t B, int64_t H, int64_t d_k,
                             int64_t d_v, int32_t L, int32_t dtype, void* stream);

/* Log-linear Gated DeltaNet forward (Sec. 3.4), with the delta-rule transition
 * alpha_t (I - beta_t k_t k_t^T) applied chunkwise through a WY (UT) representation.
 * beta is required; lambda == NULL gives plain Gated DeltaNet.  Returns LL_ERR_UNSUPPORTED
 * for shapes without a compiled kernel. */
ll_status ll_gdn_fwd(const void* q, const void* k, const void* v, const float* log_alpha,
                     const float* beta, const float* lambda, void* o, int64_t B, int64_t T,
                     int64_t H, int64_t d_k, int64_t d_v, int64_t C, int32_t dtype,
                     void* workspace, size_t workspace_bytes, void* stream);

/* Same computation as ll_gdn_fwd, for measurement: also records the caller's HIP events (as in
 * ll_mamba2_fwd_staged) on `stream`: events[0] before the per-chunk kernel, events[1] between
 * it and the level stage (the block tree of chunk transitions and states, then the per-chunk
 * read-out), events[2] after that stage.  Asynchronous.  events == NULL or any events[i] == NULL
 * returns LL_ERR_NULL_ARG. */
ll_status ll_gdn_fwd_staged(const void* q, const void* k, const void* v, const float* log_alpha,
                            const float* beta, const float* lambda, void* o, int64_t B, int64_t T,
                            int64_t H, int64_t d_k, int64_t d_v, int64_t C, int32_t dtype,
                            void* workspace, size_t workspace_bytes, void* stream,
                            void* const* events);

/* Debug: writes out[t*T + s] = the Fenwick level l(t,s) that the forward kernels assign to the
 * pair (t, s) for chunk size C (Sec. 3.1; the intra/inter split of Eq. 5), and -1 for s > t.
 * `out` is device memory of T*T bytes.  Computed on the GPU by the same device functions the
 * kernels use to pick masks and source groups, in every decomposition they use: inside a tile by
 * the tile-local indices and, for 128-row tiles, by the 16 x 16 MFMA tiles of the fast and
 * single-pass kernels; across tiles by the source-group start and by the group end.  A pair on
 * which two decompositions disagree is written as -3, a pair no source group claims as -2.
 * Requires T % C == 0, C a power of two, 1 <= T <= 16384. */
ll_status ll_debug_level_map(int64_t T, int64_t C, int8_t* out, void* stream);

/* Static, human-readable name of a status code. */
const char* ll_status_string(ll_status s);

#ifdef __cplusplus
}
#endif

#endif /* LIBLOGLINEAR_H */
