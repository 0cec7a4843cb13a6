// Host-side argument bundles and kernel tables shared by the C ABI (ll_api.hip) and the
// kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ll {

// Byte offsets of the workspace regions of one forward call (see mamba2_workspace).
struct WsLayout {
  int64_t tag = 0;     // 256 bytes: WsTag of the inputs the level summaries were formed from
  int64_t N = 0;       // tiles per sequence
  int J = 0;           // inter-tile levels
  int64_t n1 = 0, n2 = 0, nb = 0, nup = 0;  // per-(b,h) summary slots: levels 1, 2, 3 (blocks), >= 4
  int64_t tot2 = 0, t2 = 0, t3 = 0, lvl1 = 0, lvl2 = 0, blocks = 0, upper = 0, tup = 0, cnt = 0;
  int64_t tiles = 0, running = 0, cl = 0;
  int64_t total = 0;
};

// Tiles of one sequence of length T for chunk size C (the blocks the Mamba-2 kernels summarise).
int64_t tiles_of(int64_t T, int64_t C);

// Workspace layout of ll_mamba2_fwd; returns the total byte count.
int64_t mamba2_workspace(int64_t B, int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t C, int64_t esize,
                         bool has_lambda, WsLayout* lay);

// Identity of the inputs a workspace's level summaries were formed from: kept in the workspace so
// that the backward's reuse of them (ll_mamba2_bwd_after_fwd) can be checked on the device.  The
// summaries depend on the shapes, k, v and the log-gates only.
struct WsTag {
  uint64_t v[12];
};
constexpr uint64_t kWsTagMagic = 0x314741545354534CULL;  // any other value marks a workspace without summaries

struct Mamba2Args {
  const void* q;
  const void* k;
  const void* v;
  const float* log_alpha;
  const float* lambda;  // may be null
  void* o;
  int64_t B, T, H, dk, dv, C;
  int64_t Hqk;          // query/key heads (H % Hqk == 0; head h uses query/key head h / (H / Hqk))
  int L;                // Fenwick levels of T
  void* workspace;      // at least mamba2_workspace(...) bytes, 256-byte aligned
  // matrix-valued level weights (launch_ml only): [B, T, H, L, dk] diagonals or, with
  // lambda_full, [B, T, H, L, dk, dk] matrices; the workspace is mamba2_ml_workspace(...) bytes
  const float* lambda_matrix = nullptr;
  bool lambda_full = false;
  // single-pass path with lambda given: also leave the level summaries the backward reuses (the
  // workspace is at least mamba2_bwd_workspace(...) bytes)
  bool bwd_out = false;
};

typedef hipError_t (*Mamba2Launch)(const Mamba2Args&, hipStream_t, hipEvent_t* /* null or 4 events */);
constexpr int kMamba2Stages = 3;
constexpr int kMamba2MlStages = 4;  // level queries, block_state, level scan, tile_out

struct KernelEntry {
  int dtype;  // 0 = fp32, 1 = bf16
  int C, dk, dv;
  Mamba2Launch launch;
  Mamba2Launch launch_ml;  // matrix-valued level weights (null or 5 events)
};

// Workspace of the matrix-valued-weight forward: the Fenwick summaries' layout, then (full
// matrices only) the level queries [B, T, H, L, dk] at *qlev_offset; returns the total byte count.
int64_t mamba2_ml_workspace(int64_t B, int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t C, int64_t esize,
                            int L, bool full, int64_t* qlev_offset);

const KernelEntry* mamba2_table(int* n);

// The tag of the summaries formed from `a` (storage element size esize); magic = 0 gives a tag that
// matches nothing.
WsTag mamba2_tag(const Mamba2Args& a, int64_t esize, bool valid);
// Enqueues the write of `tag` into the workspace's tag region.
hipError_t launch_write_tag(void* workspace, const WsLayout& w, const WsTag& tag, hipStream_t st);
// Enqueues the write of `tag` at `dst` (a workspace's tag region).
hipError_t launch_write_tag_at(void* dst, const WsTag& tag, hipStream_t st);

// Single-pass forward (ll_mamba2_fused.hip): byte offsets of its workspace regions.
struct FusedLayout {
  int64_t N = 0;       // tiles of 128 tokens per sequence
  int J = 0;           // inter-tile levels
  int64_t stride = 0;  // floats per (b, h) row of the block sums
  // tag (at offset 0, where the three-kernel layout keeps its tag too), ticket counters, node flags,
  // block sums of the tile totals, nodes (fragment-major)
  int64_t tag = 0, ctr = 0, flag = 0, bsum = 0, node = 0;
  // with the backward's summaries: every node again in the backward's [d_v][d_k] order ([BH][N]
  // slots), the tiles' cumulative log2-gates [BH][N][128] and their totals [BH][N]
  int64_t ubwd = 0, cl = 0, t1 = 0;
  int64_t total = 0;
};
int64_t mamba2_fused_workspace(int64_t B, int64_t T, int64_t H, int64_t dk, int64_t dv, FusedLayout* lay,
                               bool bwd_out = false);
// Whether ll_mamba2_fwd takes the single-pass kernels for these arguments (dtype 1 = bf16).
bool mamba2_fused_supported(int dtype, int64_t C, int64_t dk, int64_t dv, bool has_lambda);
// Enqueues the single-pass forward; with `ev` non-null, ev[0..3] are recorded before the tile
// totals, before the block sums, before the tile kernel and after it.
hipError_t launch_mamba2_fused(const Mamba2Args& a, hipStream_t st, hipEvent_t* ev);

// Log-linear Mamba-2 backward: the forward's summary workspace followed by the key-side level
// summaries (byte offsets).
struct BwdLayout {
  WsLayout fwd;
  int64_t bad = 0;  // 256 bytes: set when the forward summaries to be reused belong to other inputs
  int64_t NR = 0, nd = 0, npart = 0;  // 8-tile regions; key-side summaries and partials per (b, h)
  int64_t d = 0, dtot = 0, part = 0, qdq = 0, tsum = 0, dqh = 0, dkh = 0, total = 0;
};
// Hqk < H adds per-head dq and dk scratch (summed over each group of heads at the end).
int64_t mamba2_bwd_workspace(int64_t B, int64_t T, int64_t H, int64_t Hqk, int64_t dk, int64_t dv, int64_t C,
                             int64_t esize, BwdLayout* lay);

struct Mamba2BwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const void* dout;
  const float* log_alpha;
  const float* lambda;
  void* dq;
  void* dk;
  void* dv;
  float* dlog_alpha;
  float* dlambda;
  int64_t B, T, H, C;
  int64_t Hqk;           // query/key heads (H % Hqk == 0); dq and dk have Hqk heads
  int L;
  void* workspace;
  bool reuse_summaries;  // the workspace already holds the forward's summaries of these inputs
  bool fused_fwd;        // ... left by the single-pass forward (FusedLayout with the backward's summaries)
};
typedef hipError_t (*Mamba2BwdLaunch)(const Mamba2BwdArgs&, hipStream_t, hipEvent_t* /* null or 5 events */);
constexpr int kMamba2BwdStages = 4;
struct BwdEntry {
  int dtype;
  int C, dk, dv;
  Mamba2BwdLaunch launch;
};
const BwdEntry* mamba2_bwd_table(int* n);

// Gated DeltaNet: per-chunk buffers carved from the workspace (byte offsets).
struct GdnLayout {
  int64_t qc = 0, pz = 0, hz = 0, oin = 0, tree = 0, total = 0;
};
int64_t gdn_workspace(int64_t B, int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t C, GdnLayout* lay);

struct GdnArgs {
  const void* q;
  const void* k;
  const void* v;
  const float* log_alpha;
  const float* beta;
  const float* lambda;  // may be null
  void* o;
  int64_t B, T, H, dk, dv, C;
  int L;
  void* workspace;
};
typedef hipError_t (*GdnLaunch)(const GdnArgs&, hipStream_t, hipEvent_t* /* null or 3 events */);
constexpr int kGdnStages = 2;
struct GdnEntry {
  int C, dk, dv;
  GdnLaunch launch;
};
const GdnEntry* gdn_table(int* n);
constexpr int kGdnMaxLevels = 16;  // inter-chunk levels of the GDN scan
hipError_t launch_debug_level_map(int64_t T, int64_t C, int8_t* out, hipStream_t st);

}  // namespace ll
