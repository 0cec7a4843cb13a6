// Single-pass log-linear Mamba-2 forward (bf16, C = 64, tiles of R = 128 tokens; lambda == NULL
// gives every level weight 1, i.e. Mamba-2 itself, through the same kernels): the chunkwise
// algorithm of Sec. 3.3 (Eq. 5; App. C, Alg. 1) with the level summaries formed and consumed
// inside one kernel, so that Q, K and V are read from HBM once.
//
// The Fenwick source groups of Sec. 3.1 are aligned blocks of tiles: tile u reads, at every set
// bit j-1 of u, the summary U_j of the 2^(j-1) tiles [((u >> (j-1)) - 1) 2^(j-1), (u >> (j-1)) 2^(j-1)).
// Every such group ends where a tile ends, and the group ending at tile e is exactly the block of
// 2^tz(e) tiles before e (tz = trailing zeros).  So each tile u publishes one "node": the summary of
// the aligned block of 2^tz(u+1) tiles that ends with u,
//     node(u) = S_u + sum over the set low bits j-1 < tz(u+1) of u of exp2(gap_j + tot_u) U_j,
// S_u = sum_t exp2(tot_u - cl_t) k_t v_t^T being the tile's own state (MFMA from its LDS-resident K
// and V) and U_j the nodes of its own low levels, which it reads anyway for its output.  Even tiles
// publish S_u alone, right after forming it; odd tiles after their intra-tile phase.
//
// Kernels, in stream order:
//   k_fused_tiles  per (tile, batch): the summed log2-gate of the tile for every head (level 0 of
//                  the block sums); clears the tiles' publication flags and the ticket counters
//   k_fused_tree   per (b, h): aligned block sums of the tile totals, levels 1 .. J-1 (the decay
//                  gaps between a tile and its source groups are sums of a few of them)
//   k_fused_fwd    per tile: the tile's state and node, the causal 128 x 128 masked contraction,
//                  and the lambda-weighted terms of every inter-tile level from the published nodes
//
// Work order and visibility.  Workgroups take tickets from the queue of the XCD they run on (the
// hardware register XCC_ID) and only from it; queue x holds the tiles of some (batch, head) pairs in
// time order (their tiles of one time step in turn), so a head's nodes are written and read through
// one L2.  With at least 64 pairs a queue holds a block of consecutive pairs, whose rows of q, k, v,
// o, lambda and the gates lie side by side in memory and share cache lines; with fewer it holds
// pairs x, x + 8, ... (measured faster there).  The grid gives every XCD as many
// workgroups as the longest queue has tiles (the hardware deals workgroups to the 8 XCDs in turn);
// a workgroup that finds its queue drained exits.  A tile only waits for nodes of earlier tickets of
// its own queue, held by workgroups that are already running, so the waits always end; each wait is
// also bounded in time (a timed-out tile writes NaN rows and counts the event).  Nodes are written
// with ordinary stores into the XCD's L2 and their flag is raised (device scope) after the stores are
// acknowledged; readers poll the flag with device-scope loads and then load the node with ordinary
// loads from the same L2.  No cache holds a node slot before it is published: every slot is written
// once per launch and never read before its flag.
//
// Latency.  Chains of odd tiles carry the nodes of large groups (node(u) waits for node(u - 1),
// node(u - 2), node(u - 4), ...), so the kernel keeps each link short: an odd tile awaits all its
// source flags first and then streams the source nodes through LDS one node ahead; K, V and the
// gates are loaded before Q so that the state, and an even tile's node, do not wait for Q; and in
// the level loop a node whose flag is not yet up is awaited after the current level's products.
#include "ll_fast_tile.hpp"
#include "ll_launch.hpp"

namespace ll {

namespace {

constexpr uint64_t kSpinTicks = 500000;  // 5 ms of the 100 MHz real-time counter
constexpr int kQueues = 8;               // XCDs of an MI355X

struct FusedWs {
  __bf16* node;    // [BH][N] node slots of DK * DV bf16, in the fragment-major MFMA result layout
  float* bsum;     // [BH][stride] aligned block sums of tile totals; level b at sum_{b'<b} ceil(N / 2^b')
  int* flag;       // [BH][N] 1 once node(u) is published
  unsigned* ctr;   // [0..7] ticket counters of the XCD queues, [8] waits that timed out
  uint64_t* tag;   // the workspace's summary tag (word 0 cleared: the backward finds no summaries)
  __bf16* ubwd;    // with the backward's summaries: [BH][N] node slots in [d_v][d_k] order
  float* cl;       //   [BH][N][R] tile-local cumulative log2-gates
  float* t1;       //   [BH][N] tile totals
  int64_t stride;
};

__device__ inline int xcc_id() {
  unsigned x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  return (int)(x & (kQueues - 1));
}

__device__ inline bool flag_up(const int* f) {
  return __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
}

// Waits until node flag *f is raised; false after kSpinTicks (the timeout is counted in *err).
__device__ inline bool wait_flag(const int* f, unsigned* err) {
  bool ok = flag_up(f);
  if (!ok) {
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    while (!(ok = flag_up(f))) {
      // about 0.5 us between polls: each poll is a device-scope load that goes to memory, and
      // denser polling (or two polls in flight) slows the publications being waited for
      __builtin_amdgcn_s_sleep(20);
      if (__builtin_amdgcn_s_memrealtime() - t0 > kSpinTicks) {
        if ((threadIdx.x & 63) == 0) __hip_atomic_fetch_add(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");  // node loads stay below the flag
  return ok;
}


// Node image layout: piece (d_k tile mk, d_v tile dv) is the 16 x 16 result block of the state
// product, 64 lanes x 4 bf16; result lane l (rows d_k = 16 mk + 4 (l / 16) + r, r = 0..3, column
// d_v = 16 dv + l % 16) is stored at slot piece_slot(l) of the piece, which puts lanes l and l + 16
// side by side, so that the 8 d_k values an operand lane needs are 16 contiguous bytes.
__device__ inline int piece_slot(int l) { return (l & 32) | ((l & 15) << 1) | ((l >> 4) & 1); }

// U^T operand fragment (d_v tile dvt, d_k step ks of 32) from a node image: slots 0-3 and 4-7 of
// the fragment (d_k 32 ks + 8 g + s) are result lanes 32 (g % 2) + i and 32 (g % 2) + 16 + i of d_k
// tile 2 ks + g / 2, i.e. slots 32 (g % 2) + 2 i and + 1: one 16-byte read.
template <int MT>
__device__ inline bf16x8 node_frag(const __bf16* img, int dvt, int ks) {
  const int lane = threadIdx.x & 63, g = lane >> 4, i = lane & 15;
  return *reinterpret_cast<const bf16x8*>(img + (((2 * ks + (g >> 1)) * MT + dvt) * 64 + 32 * (g & 1) + 2 * i) * 4);
}

// ---------------------------------------------------------------------------------------------
// Tile totals: workgroup (u, b) sums the R log2-gates of tile u for every head (16 heads at a time,
// 16 lanes per row of 16 heads).  Also clears the flags of those tiles and the ticket counters.
// ---------------------------------------------------------------------------------------------
template <int R>
__global__ __launch_bounds__(256) void k_fused_tiles(const float* __restrict__ log_alpha, FusedWs ws, int64_t Tlen,
                                                     int H, int64_t N) {
  __shared__ float part_s[4][16];
  const int64_t u = blockIdx.x;
  const int b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t row0 = (int64_t)b * Tlen + u * R;
  const int nrow = (int)((Tlen - u * R) < R ? (Tlen - u * R) : R);
  for (int h0 = 0; h0 < H; h0 += 16) {
    const int h = h0 + (tid & 15);
    // the R / 16 rows of this thread loaded together (clamped addresses, no branch), then summed in
    // row order (rows past the tile, and heads past H, add zero)
    float g[R / 16];
#pragma unroll
    for (int i = 0; i < R / 16; ++i) {
      const int r = (tid >> 4) + 16 * i;
      const bool ok = h < H && r < nrow;
      const float x = log_alpha[(row0 + (ok ? r : 0)) * H + (h < H ? h : 0)];
      g[i] = ok ? x : 0.f;
    }
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < R / 16; ++i) s += g[i] * kLog2e;
    s += __shfl_xor(s, 16, 64);
    s += __shfl_xor(s, 32, 64);
    if (lane < 16) part_s[wave][lane] = s;
    __syncthreads();
    if (tid < 16 && h0 + tid < H) {
      const int64_t bh = (int64_t)b * H + h0 + tid;
      ws.bsum[bh * ws.stride + u] = part_s[0][tid] + part_s[1][tid] + part_s[2][tid] + part_s[3][tid];
      ws.flag[bh * N + u] = 0;
    }
    __syncthreads();
  }
  if (u == 0 && b == 0 && tid < 16) ws.ctr[tid] = 0;
  if (u == 0 && b == 0 && tid == 0) ws.tag[0] = 0;  // re-tagged after the tile kernel when the backward's summaries are left
}

// ---------------------------------------------------------------------------------------------
// Block sums: workgroup bh builds levels 1 .. J-1 of the aligned block sums of its tile totals.
// Level 1 is read from level 0 in global memory; the rest are formed in LDS (dynamic, N floats).
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_fused_tree(FusedWs ws, int64_t N, int J) {
  extern __shared__ float t_s[];
  const int64_t bh = blockIdx.x;
  float* row = ws.bsum + bh * ws.stride;
  int64_t n = N, off_g = 0, off_s = 0;  // entries of the previous level; its offsets in global / LDS
  for (int b = 1; b < J; ++b) {
    const int64_t nn = (n + 1) >> 1;
    for (int64_t i = threadIdx.x; i < nn; i += blockDim.x) {
      float x;
      if (b == 1) {
        x = row[2 * i];
        if (2 * i + 1 < n) x += row[2 * i + 1];
      } else {
        x = t_s[off_s + 2 * i];
        if (2 * i + 1 < n) x += t_s[off_s + 2 * i + 1];
      }
      t_s[(b == 1 ? 0 : off_s + n) + i] = x;
      row[off_g + n + i] = x;
    }
    __syncthreads();
    if (b > 1) off_s += n;
    off_g += n;
    n = nn;
  }
}

// ---------------------------------------------------------------------------------------------
// The tile kernel.  One workgroup of 4 waves per tile (two resident per CU).  Wave w owns the
// 16-row groups w and 7 - w of the tile as in the three-kernel forward's tile kernel (O^T built
// with the query index as the MFMA column), and the d_v tiles w MT/4 .. (w + 1) MT/4 - 1 of the
// tile's state and node.
// ---------------------------------------------------------------------------------------------
template <int DK, int DV, bool HAS_LAMBDA, bool BWD_OUT>
__global__ __launch_bounds__(kFastThreads, 2) void k_fused_fwd(
    const __bf16* __restrict__ q, const __bf16* __restrict__ k, const __bf16* __restrict__ v,
    const float* __restrict__ log_alpha, const float* __restrict__ lam, FusedWs ws, __bf16* __restrict__ o,
    int64_t Tlen, int H, int Hqk, int L, int J, int64_t N, int BH) {
  using M = Mfma<__bf16>;
  typedef __bf16 bf;
  typedef typename M::frag frag;
  constexpr int R = kFastRows, LOG2R = 7;
  constexpr int NT = kFastThreads;
  constexpr int MT = DV / 16, KS = DK / M::KSTEP;
  constexpr int DKT = DK / 16, NTW = MT / 4;  // state: d_k tiles, d_v tiles per wave
  constexpr int SZ = DK * DV;
  static_assert(MT % 4 == 0 && DK <= R && DV <= R, "d_v a multiple of 64; a node fits in the K and the V region");
  __shared__ bf k_s[R * DK];
  __shared__ bf v_s[R * DV];
  __shared__ float lam_s[HAS_LAMBDA ? R * kMaxLevels : 1];
  __shared__ float cl_s[R];
  __shared__ float kdec_s[R];  // decay from each row to the end of its 16-row group
  __shared__ float tdec_s[R];  // decay from each row to the end of the tile (0 past the last row)
  __shared__ float wsum_s[4];
  __shared__ int tk_s[3];

  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  // ---- ticket from this XCD's queue
  if (tid == 0) {
    const int x = xcc_id();
    // nh pairs in queue x: first .. first + nh - 1 (BH split into 8 blocks whose sizes differ by at
    // most 1) or x, x + 8, ...
    const int base = BH / kQueues, extra = BH % kQueues;
    const int nh = base + (x < extra ? 1 : 0), first = x * base + (x < extra ? x : extra);
    const bool blocks = BH >= 8 * kQueues;
    int got = -1;
    int64_t gu = 0;
    if (nh) {
      const unsigned t = __hip_atomic_fetch_add(&ws.ctr[x], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if ((int64_t)t < (int64_t)nh * N) {
        got = blocks ? first + (int)(t % nh) : x + kQueues * (int)(t % nh);
        gu = t / nh;
      }
    }
    tk_s[0] = got;
    tk_s[1] = (int)gu;
    tk_s[2] = 0;  // set when a wait timed out
  }
  __syncthreads();
  const int bhi = __builtin_amdgcn_readfirstlane(tk_s[0]);
  if (bhi < 0) return;
  const int u = __builtin_amdgcn_readfirstlane(tk_s[1]);
  const int64_t bh = bhi;
  const int h = (int)(bh % H), b = (int)(bh / H);
  const int hq = h / (H / Hqk);
  const int64_t row0 = (int64_t)b * Tlen + (int64_t)u * R;
  const int nrow = (int)((Tlen - (int64_t)u * R) < R ? (Tlen - (int64_t)u * R) : R);
  const int gA = wave, gB = 7 - wave;
  const int iA = 16 * gA + r16, iB = 16 * gB + r16;
  const bool liveB = 16 * gB < nrow;  // nrow is a multiple of C = 64
  __bf16* node_bh = ws.node + bh * N * SZ;
  const int* flag_bh = ws.flag + bh * N;

  // ---- loads: the raw gates, lambda, K and V into LDS and the block sums of the tile's source
  //      groups (lane b: level b + 1) first; Q (into registers) once they are in, so that the
  //      state, and an even tile's node, do not wait for it
  const float la_raw = tile_gate<R>(log_alpha, row0, nrow, H, h);
  if constexpr (HAS_LAMBDA) lds_copy_lambda<R, NT>(lam_s, lam, row0, H, h, L, nrow);
  lds_copy_rows<DK, R, NT>(k_s, k + (row0 * Hqk + hq) * DK, (int64_t)Hqk * DK, nrow);
  lds_copy_rows<DV, R, NT>(v_s, v + (row0 * H + h) * DV, (int64_t)H * DV, nrow);
  float lb = 0.f;
  if (lane < J && ((u >> lane) & 1)) lb = ws.bsum[bh * ws.stride + bsum_offset(N, lane) + (u >> lane) - 1];
  auto slot_of = [&](int j) -> int64_t { return group_end(u, j) - 1; };  // node(e - 1) covers the group ending at e
  // the flags of all the tile's source groups in one poll (lane j - 1: level j); polled again after
  // the intra-tile phase, so that most levels need no poll of their own
  const bool src_lane = lane < J && ((u >> lane) & 1);
  bool fup = src_lane && flag_up(flag_bh + slot_of(lane + 1));

  // ---- gates: tile-local cumulative log2-gates, decays to the group and tile ends
  tile_cumsum_of<R>(la_raw, nrow, cl_s, wsum_s);
  for (int r = tid; r < R; r += NT) {
    kdec_s[r] = fast_exp2(cl_s[r | 15] - cl_s[r]);
    tdec_s[r] = r < nrow ? fast_exp2(cl_s[R - 1] - cl_s[r]) : 0.f;
    if constexpr (BWD_OUT) {
      ws.cl[(bh * N + u) * R + r] = cl_s[r];
      if (r == 0) ws.t1[bh * N + u] = cl_s[R - 1];
    }
  }
  // gap_j (lane j - 1): summed totals of the tile's lower-level source groups
  const float gapv = wave_inclusive_scan(lb) - lb;
  wait_vmem();
  __syncthreads();  // K, V, lambda, decays visible
  frag qA[KS], qB[KS];
  {
    const int rA = iA < nrow ? iA : nrow - 1, rB = iB < nrow ? iB : nrow - 1;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      qA[ks] = M::load(q + ((row0 + rA) * Hqk + hq) * DK + ks * M::KSTEP + g * M::KPL);
      qB[ks] = liveB ? M::load(q + ((row0 + rB) * Hqk + hq) * DK + ks * M::KSTEP + g * M::KPL) : frag{};
    }
  }

  // ---- the tile's state S_u = K^T diag(tdec) V: d_k x (this wave's d_v tiles), K = R tokens
  bf16x4 sbf[DKT][NTW];
  {
    f32x4 sacc[DKT][NTW];
#pragma unroll
    for (int mt = 0; mt < DKT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt) sacc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ts = 0; ts < R / 32; ++ts) {
      const f32x4 d0 = *reinterpret_cast<const f32x4*>(&tdec_s[32 * ts + 4 * g]);
      const f32x4 d1 = *reinterpret_cast<const f32x4*>(&tdec_s[32 * ts + 16 + 4 * g]);
      frag vb[NTW];
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt) {
        frag x = frag_down_rows_swz<DV>(v_s, 32 * ts, 16 * (wave * NTW + nt));
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          x[s] = from_f32<bf>(to_f32(x[s]) * d0[s]);
          x[4 + s] = from_f32<bf>(to_f32(x[4 + s]) * d1[s]);
        }
        vb[nt] = x;
      }
#pragma unroll
      for (int mt = 0; mt < DKT; ++mt) {
        const frag a = frag_down_rows_swz<DK>(k_s, 32 * ts, 16 * mt);
#pragma unroll
        for (int nt = 0; nt < NTW; ++nt) sacc[mt][nt] = M::mma(a, vb[nt], sacc[mt][nt]);
      }
    }
#pragma unroll
    for (int mt = 0; mt < DKT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt)
#pragma unroll
        for (int r = 0; r < 4; ++r) sbf[mt][nt][r] = from_f32<bf>(sacc[mt][nt][r]);
  }
  // node(u) pieces of this wave: write-through stores, then (after every wave's) the flag
  auto publish = [&]() {
    bf* dst = node_bh + (int64_t)u * SZ;
#pragma unroll
    for (int mt = 0; mt < DKT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt)
        *reinterpret_cast<bf16x4*>(dst + ((mt * MT + wave * NTW + nt) * 64 + piece_slot(lane)) * 4) = sbf[mt][nt];
    wait_vmem();
    __syncthreads();
    if (tid == 0) __hip_atomic_store(ws.flag + bh * N + u, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if constexpr (BWD_OUT) {  // the same pieces in the backward's order (row d_v, four consecutive d_k)
      bf* ub = ws.ubwd + (bh * N + u) * SZ;
#pragma unroll
      for (int mt = 0; mt < DKT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTW; ++nt)
          *reinterpret_cast<bf16x4*>(ub + (16 * (wave * NTW + nt) + r16) * DK + 16 * mt + 4 * g) = sbf[mt][nt];
    }
  };
  if (!(u & 1)) publish();

  // ---- intra-tile: causal 128 x 128 masked contraction
  const float cliA = cl_s[iA], cliB = cl_s[iB];
  const float* lrowA = &lam_s[HAS_LAMBDA ? iA * kMaxLevels : 0];
  const float* lrowB = &lam_s[HAS_LAMBDA ? iB * kMaxLevels : 0];
  f32x4 oA[MT], oB[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) oA[mt] = oB[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  fast_intra<DK, DV, HAS_LAMBDA>(wave, k_s, v_s, cl_s, kdec_s, qA, qB, cliA, cliB, lrowA, lrowB, oA, oB);
  if (src_lane && !fup) fup = flag_up(flag_bh + slot_of(lane + 1));
  const uint64_t seen = __ballot(fup);  // bit j - 1: node of level j known to be published
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");  // node loads stay below the polls
  auto await_level = [&](int j) {
    if (!((seen >> (j - 1)) & 1) && !wait_flag(flag_bh + slot_of(j), ws.ctr + 8)) tk_s[2] = 1;
  };

  // ---- odd tiles: node(u) = S_u + the tile's low-level groups, decayed to the end of the tile.
  //      Every source flag is awaited first; then each wave streams its own pieces of the source
  //      nodes through two slots of its own in the (now free) K and V regions, one node ahead.
  if (u & 1) {
    const int t = __builtin_ctz(~(unsigned)u);  // levels 1..t: the low set bits of u
    const float tot_u = cl_s[R - 1];
    f32x4 acc[DKT][NTW];
#pragma unroll
    for (int mt = 0; mt < DKT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[mt][nt][r] = to_f32(sbf[mt][nt][r]);
    for (int j = 1; j <= t; ++j) await_level(j);
    __syncthreads();  // every wave is done with K and V
    // slot x of this wave: SLICE bf16 = its pieces (d_k tile mt, d_v tile nt) at (mt NTW + nt) 256
    constexpr int SLICE = DKT * NTW * 256, PCS = SLICE / 8, NPW = PCS / 64;
    bf* const slots = (wave < 2 ? k_s : v_s) + (wave & 1) * 2 * SLICE;
    auto issue = [&](int jj, bf* dst) {
      const bf* src = node_bh + slot_of(jj) * SZ + wave * NTW * 256;
#pragma unroll
      for (int i = 0; i < NPW; ++i) {
        const int pq = i * 64 + lane, mt = pq / (NTW * 32), rem = pq % (NTW * 32);
        __builtin_amdgcn_global_load_lds(src + mt * MT * 256 + rem * 8,
                                         (__attribute__((address_space(3))) void*)(dst + i * 512), 16, 0, 0);
      }
    };
    issue(1, slots);
    for (int j = 1; j <= t; ++j) {
      if (j < t) {
        issue(j + 1, slots + (j & 1) * SLICE);
        wait_vmcnt<NPW>();
      } else {
        wait_vmcnt<0>();
      }
      const float w = fast_exp2(gap_of(gapv, j) + tot_u);
      const bf* cur = slots + ((j - 1) & 1) * SLICE;
#pragma unroll
      for (int mt = 0; mt < DKT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTW; ++nt) {
          const bf16x4 pc = *reinterpret_cast<const bf16x4*>(cur + (mt * NTW + nt) * 256 + piece_slot(lane) * 4);
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[mt][nt][r] += w * to_f32(pc[r]);
        }
    }
#pragma unroll
    for (int mt = 0; mt < DKT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt)
#pragma unroll
        for (int r = 0; r < 4; ++r) sbf[mt][nt][r] = from_f32<bf>(acc[mt][nt][r]);
    publish();
  }

  // ---- inter-tile levels: the set bits of u, highest (oldest node) first; the nodes alternate
  //      between the K and V regions, the next one copied in while the current one is used
  auto copy_node = [&](int j, bf* dst) {
    const bf* src = node_bh + slot_of(j) * SZ;
    lds_gather16<NT>(dst, SZ * 2 / 16, [&](int x) { return src + 8 * x; });
  };
  auto copy_level = [&](int j, bf* dst) {
    await_level(j);
    copy_node(j, dst);
  };
  auto next_level = [&](int j) {
    for (--j; j >= 1; --j)
      if ((u >> (j - 1)) & 1) return j;
    return 0;
  };
  // lambda == NULL (every level weight 1): the row factor exp2(c_t) comes out of the level sum, so
  // the tile sums its source nodes, each weighted by exp2(gap_j), into this wave's pieces of one
  // fp32 state and multiplies Q by that state once after the loop, instead of once per level.  The
  // sum is elementwise, so lane l sums slot l of each piece (consecutive 8-byte reads) and writes
  // the result back to slot l
  f32x4 pre[DKT][NTW];
  if constexpr (!HAS_LAMBDA) {
#pragma unroll
    for (int mt = 0; mt < DKT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt) pre[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  auto level_step = [&](int& j, const bf* cur, bf* nxt) {
    wait_vmem();
    __syncthreads();  // `cur` complete and visible; every wave is done with `nxt`
    const int jn = next_level(j);
    // a node not yet published is awaited after this level's products, not before them
    const bool early = jn && (((seen >> (jn - 1)) & 1) || flag_up(flag_bh + slot_of(jn)));
    if (early) {
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      copy_node(jn, nxt);
    }
    const float gap = gap_of(gapv, j);
    if constexpr (HAS_LAMBDA) {
      const float wA = fast_exp2(cliA + gap) * lrowA[LOG2R + j], wB = fast_exp2(cliB + gap) * lrowB[LOG2R + j];
      frag uf[2][KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) uf[0][ks] = node_frag<MT>(cur, 0, ks);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        if (mt + 1 < MT) {
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) uf[(mt + 1) & 1][ks] = node_frag<MT>(cur, mt + 1, ks);
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
    } else {
      const float w = fast_exp2(gap);
#pragma unroll
      for (int mt = 0; mt < DKT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTW; ++nt) {
          const bf16x4 pc = *reinterpret_cast<const bf16x4*>(cur + ((mt * MT + wave * NTW + nt) * 64 + lane) * 4);
#pragma unroll
          for (int r = 0; r < 4; ++r) pre[mt][nt][r] += w * to_f32(pc[r]);
        }
    }
    if (jn && !early) copy_level(jn, nxt);
    j = jn;
  };
  int j = u ? bitlen((uint32_t)u) : 0;
  __syncthreads();  // every wave is done with K and V
  if (j) copy_level(j, k_s);
  while (j) {
    level_step(j, k_s, v_s);
    if (!j) break;
    level_step(j, v_s, k_s);
  }
  if constexpr (!HAS_LAMBDA) {
    if (u) {  // the combined state (bf16, node layout) into the K region, then one product pass
      __syncthreads();  // every wave is done with the last node
#pragma unroll
      for (int mt = 0; mt < DKT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NTW; ++nt) {
          bf16x4 v4;
#pragma unroll
          for (int r = 0; r < 4; ++r) v4[r] = from_f32<bf>(pre[mt][nt][r]);
          *reinterpret_cast<bf16x4*>(k_s + ((mt * MT + wave * NTW + nt) * 64 + lane) * 4) = v4;
        }
      __syncthreads();
      const float wA = fast_exp2(cliA), wB = fast_exp2(cliB);
      frag uf[2][KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) uf[0][ks] = node_frag<MT>(k_s, 0, ks);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        if (mt + 1 < MT) {
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) uf[(mt + 1) & 1][ks] = node_frag<MT>(k_s, mt + 1, ks);
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
    }
  }

  // ---- store O through LDS (rows iA, iB staged into a swizzled row-major tile in the V region)
  __syncthreads();  // every wave is done with the last node; tk_s[2] final
  const bool failed = tk_s[2] != 0;
  auto stage_rows = [&](const f32x4* acc, int i) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      bf16x4 val;
#pragma unroll
      for (int r = 0; r < 4; ++r) val[r] = from_f32<bf>(failed ? __builtin_nanf("") : acc[mt][r]);
      *reinterpret_cast<bf16x4*>(v_s + swz<DV>(i, 2 * mt + (g >> 1)) + 4 * (g & 1)) = val;
    }
  };
  stage_rows(oA, iA);
  stage_rows(oB, iB);
  __syncthreads();
  constexpr int OCH = DV / 8;
#pragma unroll
  for (int it = 0; it < R * OCH / NT; ++it) {
    const int idx = it * NT + tid, r = idx / OCH, c = idx % OCH;
    if (r < nrow)
      *reinterpret_cast<bf16x8*>(o + ((row0 + r) * H + h) * DV + 8 * c) = *reinterpret_cast<const bf16x8*>(v_s + swz<DV>(r, c));
  }
}

}  // namespace

int64_t mamba2_fused_workspace(int64_t B, int64_t T, int64_t H, int64_t dk, int64_t dv, FusedLayout* lay,
                               bool bwd_out) {
  auto al = [](int64_t x) { return (x + 255) & ~int64_t(255); };
  FusedLayout w;
  w.N = tiles_of(T, 64);
  w.J = w.N <= 1 ? 0 : 64 - __builtin_clzll(uint64_t(w.N - 1));
  w.stride = bsum_offset(w.N, w.J > 1 ? w.J : 1);
  const int64_t BH = B * H;
  int64_t cur = 0;
  w.tag = cur; cur += al(sizeof(WsTag));
  w.ctr = cur; cur += al(16 * 4);
  w.flag = cur; cur += al(BH * w.N * 4);
  w.bsum = cur; cur += al(BH * w.stride * 4);
  w.node = cur; cur += al(BH * w.N * dk * dv * 2);
  if (bwd_out) {
    w.ubwd = cur; cur += al(BH * w.N * dk * dv * 2);
    w.cl = cur; cur += al(BH * w.N * kFastRows * 4);
    w.t1 = cur; cur += al(BH * w.N * 4);
  }
  w.total = cur;
  if (lay) *lay = w;
  return cur;
}

bool mamba2_fused_supported(int dtype, int64_t C, int64_t dk, int64_t dv, bool has_lambda) {
  (void)has_lambda;  // lambda == NULL runs the same kernels with every level weight 1
  return dtype == 1 && C == 64 && (dk == 64 || dk == 128) && (dv == 64 || dv == 128);
}

template <int DK, int DV>
static hipError_t launch_fused(const Mamba2Args& a, hipStream_t st, hipEvent_t* ev) {
  const bool bwd_out = a.bwd_out && a.lambda;
  FusedLayout w;
  mamba2_fused_workspace(a.B, a.T, a.H, DK, DV, &w, bwd_out);
  char* base = static_cast<char*>(a.workspace);
  FusedWs ws;
  ws.node = reinterpret_cast<__bf16*>(base + w.node);
  ws.bsum = reinterpret_cast<float*>(base + w.bsum);
  ws.flag = reinterpret_cast<int*>(base + w.flag);
  ws.ctr = reinterpret_cast<unsigned*>(base + w.ctr);
  ws.tag = reinterpret_cast<uint64_t*>(base + w.tag);
  ws.ubwd = reinterpret_cast<__bf16*>(base + w.ubwd);
  ws.cl = reinterpret_cast<float*>(base + w.cl);
  ws.t1 = reinterpret_cast<float*>(base + w.t1);
  ws.stride = w.stride;
  const int BH = (int)(a.B * a.H);
  if (ev) (void)hipEventRecord(ev[0], st);
  hipLaunchKernelGGL((k_fused_tiles<kFastRows>), dim3((unsigned)w.N, (unsigned)a.B), dim3(256), 0, st, a.log_alpha, ws,
                     a.T, (int)a.H, w.N);
  if (ev) (void)hipEventRecord(ev[1], st);
  if (w.J > 1) {
    const int64_t n1 = (w.N + 1) / 2;  // the largest level formed in LDS
    hipLaunchKernelGGL(k_fused_tree, dim3((unsigned)BH), dim3(256), (size_t)n1 * 2 * sizeof(float), st, ws, w.N, w.J);
  }
  if (ev) (void)hipEventRecord(ev[2], st);
  // every XCD receives (workgroups round-robin) as many workgroups as its queue has tiles
  const int64_t grid = (int64_t)kQueues * ((BH + kQueues - 1) / kQueues) * w.N;
  if (bwd_out)
    hipLaunchKernelGGL((k_fused_fwd<DK, DV, true, true>), dim3((unsigned)grid), dim3(kFastThreads), 0, st,
                       (const __bf16*)a.q, (const __bf16*)a.k, (const __bf16*)a.v, a.log_alpha, a.lambda, ws,
                       (__bf16*)a.o, a.T, (int)a.H, (int)a.Hqk, a.L, w.J, w.N, BH);
  else if (a.lambda)
    hipLaunchKernelGGL((k_fused_fwd<DK, DV, true, false>), dim3((unsigned)grid), dim3(kFastThreads), 0, st,
                       (const __bf16*)a.q, (const __bf16*)a.k, (const __bf16*)a.v, a.log_alpha, a.lambda, ws,
                       (__bf16*)a.o, a.T, (int)a.H, (int)a.Hqk, a.L, w.J, w.N, BH);
  else
    hipLaunchKernelGGL((k_fused_fwd<DK, DV, false, false>), dim3((unsigned)grid), dim3(kFastThreads), 0, st,
                       (const __bf16*)a.q, (const __bf16*)a.k, (const __bf16*)a.v, a.log_alpha, a.lambda, ws,
                       (__bf16*)a.o, a.T, (int)a.H, (int)a.Hqk, a.L, w.J, w.N, BH);
  // the summaries the backward reuses are complete: tag them with the inputs they came from
  if (bwd_out) {
    const hipError_t e = launch_write_tag_at(ws.tag, mamba2_tag(a, 2, true), st);
    if (e != hipSuccess) return e;
  }
  if (ev) (void)hipEventRecord(ev[3], st);
  return hipGetLastError();
}

hipError_t launch_mamba2_fused(const Mamba2Args& a, hipStream_t st, hipEvent_t* ev) {
  if (a.dk == 128 && a.dv == 128) return launch_fused<128, 128>(a, st, ev);
  if (a.dk == 128 && a.dv == 64) return launch_fused<128, 64>(a, st, ev);
  if (a.dk == 64 && a.dv == 64) return launch_fused<64, 64>(a, st, ev);
  if (a.dk == 64 && a.dv == 128) return launch_fused<64, 128>(a, st, ev);
  return hipErrorInvalidValue;
}

}  // namespace ll
