// Host-side argument bundles and kernel tables shared by the C ABI (ll_api.hip) and the
// kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ll {

// Workspace regions, carved by the C ABI from the caller's buffer (all device pointers).
struct Workspace {
  float* tot2 = nullptr;      // [B*H][N]          chunk totals of log2-domain gates
  float* gaps2 = nullptr;     // [B*H][N][J]       log2 decay from a source group's end to a reader
  float* states = nullptr;    // [B*H][N][d_v*d_k] chunk states, fp32, layout [p][n]
  void* nodes = nullptr;      // [B*H][nodes_per_bh][d_v*d_k] level summaries (storage dtype)
  int64_t nodes_per_bh = 0;
};

struct Mamba2Args {
  const void* q;
  const void* k;
  const void* v;
  const float* log_alpha;
  const float* lambda;  // may be null
  void* o;
  int64_t B, T, H, dk, dv, C;
  int L;  // Fenwick levels of T
  int J;  // inter-chunk levels
  Workspace ws;
};

typedef hipError_t (*Mamba2Launch)(const Mamba2Args&, hipStream_t, hipEvent_t* /* null or 4 events */);
constexpr int kMamba2Stages = 3;

struct KernelEntry {
  int dtype;  // 0 = fp32, 1 = bf16
  int C, dk, dv;
  Mamba2Launch launch;
};

const KernelEntry* mamba2_table(int* n);
hipError_t launch_debug_level_map(int64_t T, int C, int log2C, int J, int8_t* out, hipStream_t st);

}  // namespace ll
