// Intra-tile building block of the bf16 tile kernels with R = 128 rows (C = 64): the causal
// 128 x 128 masked contraction of Eq. 5's diagonal blocks plus the lowest inter-chunk level, with
// the tile's K and V resident in swizzled LDS tiles and its Q in registers.  Shared by the
// three-kernel forward (ll_mamba2.hip) and the single-pass forward (ll_mamba2_fused.hip).
#pragma once

#include <type_traits>

#include "ll_mamba2_common.hpp"

namespace ll {

constexpr int kFastRows = 128;
constexpr int kFastThreads = 256;

// Intra-tile part of the 128-row fast kernels: causal 128 x 128 masked contraction of the
// tile's Q (registers: rows iA = 16 wave + r16 and iB = 16 (7 - wave) + r16 of this lane) with
// its K and V (swizzled LDS tiles), 32 keys per step, no barrier.  The body is instantiated per
// wave (groups GA = wave, GB = 7 - wave known at compile time), so that every skipped key tile
// and every mask case is resolved statically.  Accumulates into oA, oB (O^T fragments).
//
// MTW d_v tiles starting at tile mt0 are accumulated (all DV / 16 of them by default); a wave
// that covers only part of d_v still forms the full score tiles of its rows.
template <int DK, int DV, bool HAS_LAMBDA, int MTW = DV / 16>
__device__ __attribute__((always_inline)) inline void fast_intra(
    int wave, const __bf16* k_s, const __bf16* v_s, const float* cl_s, const float* kdec_s,
    const bf16x8 (&qA)[DK / 32], const bf16x8 (&qB)[DK / 32], float cliA, float cliB, const float* lrowA,
    const float* lrowB, f32x4 (&oA)[MTW], f32x4 (&oB)[MTW], int mt0 = 0) {
  using M = Mfma<__bf16>;
  typedef __bf16 bf;
  typedef typename M::frag frag;
  constexpr int KS = DK / M::KSTEP, KC = M::KSTEP / 8;
  const int lane = threadIdx.x & 63, r16 = lane & 15, g = lane >> 4;
  // weights of the diagonal 16 x 16 tile (keys 16 gi + 4g + r): decay and lambda of the level
  // bitlen(r16 ^ (4g + r)); zero above the diagonal
  auto diag_weights = [&](int gi, float cli, const float* lrow) {
    f32x4 w;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int jl = 4 * g + r;
      float x = fast_exp2(fminf(cli - cl_s[16 * gi + jl], 0.f));
      if constexpr (HAS_LAMBDA) x *= lrow[level_in_group(r16, jl)];
      w[r] = jl <= r16 ? x : 0.f;
    }
    return w;
  };
  // off-diagonal key tile KT < gi: one level for the whole tile, decay split at its last key
  auto offdiag = [&](f32x4 sacc, int KT, int gi, float cli, const float* lrow) {
    float qs = fast_exp2(cli - cl_s[16 * KT + 15]);
    if constexpr (HAS_LAMBDA) qs *= lrow[level_across_groups(gi, KT)];
    const f32x4 kd = *reinterpret_cast<const f32x4*>(&kdec_s[16 * KT + 4 * g]);
    f32x4 p;
#pragma unroll
    for (int r = 0; r < 4; ++r) p[r] = sacc[r] * qs * kd[r];
    return p;
  };

  auto intra = [&](auto wave_c) {
    constexpr int GA = decltype(wave_c)::value, GB = 7 - GA;
    const f32x4 wdA = diag_weights(GA, cliA, lrowA), wdB = diag_weights(GB, cliB, lrowB);
    auto mask = [&](f32x4 sacc, auto kt_c, auto gi_c, float cli, const float* lrow, f32x4 wd) {
      constexpr int KT = decltype(kt_c)::value, GI = decltype(gi_c)::value;
      if constexpr (KT < GI) {
        return offdiag(sacc, KT, GI, cli, lrow);
      } else if constexpr (KT == GI) {
        f32x4 p;
#pragma unroll
        for (int r = 0; r < 4; ++r) p[r] = sacc[r] * wd[r];
        return p;
      } else {
        return f32x4{0.f, 0.f, 0.f, 0.f};
      }
    };
    auto step = [&](auto st_c) {
      constexpr int ST = decltype(st_c)::value, KT0 = 2 * ST, KT1 = 2 * ST + 1;
      constexpr bool B0 = KT0 <= GB, B1 = KT1 <= GB, A0 = KT0 <= GA, A1 = KT1 <= GA;
      if constexpr (B0) {  // GB > GA: group B reaches every key tile group A does
        f32x4 sA0 = {0.f, 0.f, 0.f, 0.f}, sA1 = sA0, sB0 = sA0, sB1 = sA0;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const frag k0 = frag_along_row_swz<DK>(k_s, 16 * KT0, ks * KC);
          sB0 = M::mma(k0, qB[ks], sB0);
          if constexpr (A0) sA0 = M::mma(k0, qA[ks], sA0);
          if constexpr (B1) {
            const frag k1 = frag_along_row_swz<DK>(k_s, 16 * KT1, ks * KC);
            sB1 = M::mma(k1, qB[ks], sB1);
            if constexpr (A1) sA1 = M::mma(k1, qA[ks], sA1);
          }
        }
        // P^T fragments: slots 0-3 <- key tile KT0 rows 4g..4g+3, slots 4-7 <- key tile KT1
        frag pA, pB;
        {
          using K0 = std::integral_constant<int, KT0>;
          using K1 = std::integral_constant<int, KT1>;
          using CA = std::integral_constant<int, GA>;
          using CB = std::integral_constant<int, GB>;
          const f32x4 m0 = mask(sB0, K0{}, CB{}, cliB, lrowB, wdB), m1 = mask(sB1, K1{}, CB{}, cliB, lrowB, wdB);
          const f32x4 n0 = mask(sA0, K0{}, CA{}, cliA, lrowA, wdA), n1 = mask(sA1, K1{}, CA{}, cliA, lrowA, wdA);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            pB[r] = from_f32<bf>(m0[r]);
            pB[4 + r] = from_f32<bf>(m1[r]);
            pA[r] = from_f32<bf>(n0[r]);
            pA[4 + r] = from_f32<bf>(n1[r]);
          }
        }
#pragma unroll
        for (int mt = 0; mt < MTW; ++mt) {
          const frag vf = frag_down_rows_swz<DV>(v_s, ST * 32, (mt0 + mt) * 16);
          oB[mt] = M::mma(vf, pB, oB[mt]);
          if constexpr (A0) oA[mt] = M::mma(vf, pA, oA[mt]);
        }
      }
    };
    step(std::integral_constant<int, 0>{});
    step(std::integral_constant<int, 1>{});
    step(std::integral_constant<int, 2>{});
    step(std::integral_constant<int, 3>{});
  };
  switch (wave) {
    case 0: intra(std::integral_constant<int, 0>{}); break;
    case 1: intra(std::integral_constant<int, 1>{}); break;
    case 2: intra(std::integral_constant<int, 2>{}); break;
    default: intra(std::integral_constant<int, 3>{}); break;
  }

}

}  // namespace ll
