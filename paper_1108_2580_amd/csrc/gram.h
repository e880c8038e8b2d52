// Device building blocks shared by the row kernels: lane layout helpers and
// the gather + MFMA accumulation of one item's normal equations (Sec. 2.2)
// together with the squared residuals of the entering state (Sec. 4.1).
//
// Lane (kq, c) = (lane / 16, lane % 16). Operand block X of rating k is
// feature 16 X + c of the staged fixed row f_k in lane (k, c); one
// v_mfma_f32_16x16x4f32 consumes four ratings. Accumulator tile (I, J),
// I <= J, holds G[16 I + 4 kq + r][16 J + c] in element r.
#pragma once

#include "internal.h"

namespace als {

typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ float swz_xor(float v, int x) {
  // ds_swizzle bit mode: lane' = lane ^ x within 32-lane halves
  switch (x) {
    case 1: return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x041F));
    case 2: return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x081F));
    case 4: return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x101F));
    default: return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x201F));
  }
}

// Rotate a value right by K lanes within each 16-lane row (DPP row_ror).
template <int K>
__device__ __forceinline__ float row_ror(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x120 + K, 0xF, 0xF, false));
}

// Sum over the 16 lanes of a row; every lane of the row receives the same value.
__device__ __forceinline__ float sum16(float v) {
  v += row_ror<8>(v);
  v += row_ror<4>(v);
  v += row_ror<2>(v);
  v += row_ror<1>(v);
  return v;
}

// Value of lane l (wave-uniform) broadcast to the wave through a scalar register.
__device__ __forceinline__ float lane_value(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

// 1 / sqrt(p) of a pivot, clamped to a small positive value (callers flag pivots that
// are not positive and finite). The hardware reciprocal square root is accurate to
// about one ulp; the exactly rounded sqrtf and division cost about 25 dependent
// instructions per pivot on the factorisation's critical path.
__device__ __forceinline__ float inv_sqrt_pivot(float p) {
  return __builtin_amdgcn_rsqf(fmaxf(p, 1e-30f));
}

template <int T>
__host__ __device__ constexpr int tidx(int I, int J) {
  return I * T - I * (I - 1) / 2 + (J - I);
}

template <int DP>
struct RowCfg {
  static constexpr int T = DP / 16;
  static constexpr int NT = T * (T + 1) / 2;
  // steps per gathered block (wide rows keep two blocks in flight)
  static constexpr int STEPS = T <= 2 ? 16 : (T <= 4 ? 8 : (T <= 6 ? 4 : 2));
};

template <int V>
struct IntC {
  static constexpr int value = V;
};

template <int B, int NB, class F>
__device__ __forceinline__ void unroll_blocks(F &f) {
  if constexpr (B < NB) {
    f(IntC<B>{});
    unroll_blocks<B + 1, NB>(f);
  }
}

// Gather the staged fixed rows of steps s0 .. s0 + STEPS - 1 of a 64-rating group:
// lane (kq, c) receives feature 16 X + c of rating 4 s + kq. jsrc / rsrc hold the
// group's column indices and ratings, one per lane.
// Loads are never predicated per lane (a predicated load becomes a branch that waits
// for its own completion, which serialises the gathers): ratings past the end of the
// item read the staged all-zero row, and padded features read the staged row's zero
// padding. One 32-bit byte offset per step from the (uniform) table base; the tiles
// follow at immediate offsets.
// With AUG, lane column aug_c of the last tile carries the rating instead of the
// (zero) padded feature, so that the MFMA Gram also accumulates b = sum r f in that
// column (and sum r^2 on its diagonal).
template <int DP, int STEPS, bool AUG>
__device__ __forceinline__ void gather_block(float (&a)[STEPS][DP / 16], float (&r)[STEPS],
                                             int jsrc, float rsrc, int s0,
                                             const float *__restrict__ Fp, bool aug_lane) {
  constexpr int T = DP / 16;
  const int lane = threadIdx.x & 63;
  const int kq = lane >> 4, c = lane & 15;
#pragma unroll
  for (int u = 0; u < STEPS; ++u) {
    const int src = 4 * (s0 + u) + kq;
    const int j = __shfl(jsrc, src);
    r[u] = __shfl(rsrc, src);
    const uint32_t off = (uint32_t)j * (uint32_t)(DP * 4) + (uint32_t)(c * 4);
    const char *row = reinterpret_cast<const char *>(Fp) + (uint64_t)off;
#pragma unroll
    for (int X = 0; X < T; ++X) a[u][X] = *reinterpret_cast<const float *>(row + 64 * X);
    if constexpr (AUG) a[u][T - 1] = aug_lane ? r[u] : a[u][T - 1];
  }
}

// MFMA Gram update, right-hand side and per-step partial predictions of the gathered
// steps s0 .. s0 + STEPS - 1, in sub-blocks of up to four steps; sub-blocks past the
// item's last step (steps of this group) are skipped. With AUG the right-hand side is
// a column of the Gram and rhs is left alone.
template <int DP, int STEPS, bool AUG>
__device__ __forceinline__ void mma_block(floatx4 (&acc)[RowCfg<DP>::NT],
                                          float (&rhs)[DP / 16], const float (&xo)[DP / 16],
                                          float (&pi)[16], const float (&a)[STEPS][DP / 16],
                                          const float (&r)[STEPS], int s0, int steps) {
  constexpr int T = DP / 16, SUB = STEPS < 4 ? STEPS : 4;
#pragma unroll
  for (int u0 = 0; u0 < STEPS; u0 += SUB) {
    if (s0 + u0 < steps) {
#pragma unroll
      for (int u = u0; u < u0 + SUB; ++u) {
#pragma unroll
        for (int X = 0; X < T; ++X) {
          if constexpr (!AUG) rhs[X] = fmaf(r[u], a[u][X], rhs[X]);
          pi[s0 + u] = fmaf(a[u][X], xo[X], pi[s0 + u]);
        }
#pragma unroll
        for (int I = 0; I < T; ++I) {
#pragma unroll
          for (int J = I; J < T; ++J)
            acc[tidx<T>(I, J)] =
                __builtin_amdgcn_mfma_f32_16x16x4f32(a[u][I], a[u][J], acc[tidx<T>(I, J)], 0, 0, 0);
        }
      }
    }
  }
}

// End of a 64-rating group: reduce-scatter the 16 step partials over the 16 feature
// lanes, after which lane c holds the full prediction of step c for its rating group
// (both halves are exchanged and the lane keeps the sum of its half; selecting between
// computed sums keeps the partial array statically indexed), and add the squared
// residuals of the group's ratings.
__device__ __forceinline__ void group_residuals(float (&pi)[16], float rv, int g, int n,
                                                double &sse) {
  const int lane = threadIdx.x & 63;
  const int kq = lane >> 4, c = lane & 15;
#pragma unroll
  for (int o = 8, m = 16; o >= 1; o >>= 1, m >>= 1) {
    const bool hi = (c & o) != 0;
#pragma unroll
    for (int i = 0; i < m / 2; ++i) {
      const float lo_sum = pi[i] + swz_xor(pi[i], o);
      const float hi_sum = pi[m / 2 + i] + swz_xor(pi[m / 2 + i], o);
      pi[i] = hi ? hi_sum : lo_sum;
    }
  }
  // lane (kq, c) now holds the prediction of rating g + 4c + kq, whose value sits in
  // lane 4c + kq of this group's rating register
  const float rq = __shfl(rv, 4 * c + kq);
  if (g + 4 * c + kq < n) {
    const double e = (double)rq - (double)pi[0];
    sse = fma(e, e, sse);
  }
}

// Accumulate the item's Gram tiles and right-hand side and the entering-state squared
// residuals. Without AUG the right-hand side is kept in rhs as per-lane partials over
// the four rating groups; with AUG it is the Gram's column 16 (T - 1) + aug_c (a padding
// column whose lane carries the ratings) and rhs is untouched.
// xo: the row's current factor values in lane-column form (xo[X] = x[16X + c]).
// Ratings are taken in groups of 64, each gathered in blocks of STEPS steps (four
// ratings per step).
//  - Narrow rows (T <= 2): one block per group, gathered and then multiplied.
//  - Wider rows: two block buffers; the gather of the next block (of this group, or
//    the first block of the next group) is issued before the MFMAs of the current
//    one, so that its latency hides behind them. The blocks of the last group that
//    lie past the item's end are still gathered (from the zero row) but not multiplied.
template <int DP, bool AUG>
__device__ __forceinline__ void gram_accumulate(floatx4 (&acc)[RowCfg<DP>::NT],
                                                float (&rhs)[RowCfg<DP>::T],
                                                const float (&xo)[RowCfg<DP>::T], double &sse,
                                                const int32_t *__restrict__ ip,
                                                const uint8_t *__restrict__ vp, int n,
                                                const float *__restrict__ Fp, int zrow,
                                                int aug_c) {
  using C = RowCfg<DP>;
  constexpr int T = C::T, STEPS = C::STEPS, NB = 16 / STEPS;
  const int lane = threadIdx.x & 63;
  const bool aug_lane = (lane & 15) == aug_c;
  int jv = lane < n ? ip[lane] : zrow;
  float rv = (float)vp[min(lane, n - 1)];
  rv = lane < n ? rv : 0.f;
  if constexpr (T <= 2) {
    for (int g = 0; g < n; g += 64) {
      const int gn = g + 64 + lane;
      const int jl = ip[min(gn, n - 1)];
      const float rl = (float)vp[min(gn, n - 1)];
      const int jn = gn < n ? jl : zrow;
      const float rn = gn < n ? rl : 0.f;
      const int steps = min(16, (n - g + 3) >> 2);
      __builtin_assume(steps >= 1);  // g < n: the group's first step always exists
      float pi[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) pi[u] = 0.f;
#pragma unroll
      for (int s0 = 0; s0 < 16; s0 += STEPS) {
        if (s0 < steps) {
          float a[STEPS][T];
          float r[STEPS];
          gather_block<DP, STEPS, AUG>(a, r, jv, rv, s0, Fp, aug_lane);
          mma_block<DP, STEPS, AUG>(acc, rhs, xo, pi, a, r, s0, steps);
        }
      }
      group_residuals(pi, rv, g, n, sse);
      jv = jn;
      rv = rn;
    }
  } else {
    static_assert(NB % 2 == 0, "block buffers alternate within and across groups");
    float a0[STEPS][T], a1[STEPS][T], r0[STEPS], r1[STEPS];
    gather_block<DP, STEPS, AUG>(a0, r0, jv, rv, 0, Fp, aug_lane);
    for (int g = 0; g < n; g += 64) {
      const int gn = g + 64 + lane;
      const int jl = ip[min(gn, n - 1)];
      const float rl = (float)vp[min(gn, n - 1)];
      const int jn = gn < n ? jl : zrow;
      const float rn = gn < n ? rl : 0.f;
      const int steps = min(16, (n - g + 3) >> 2);
      __builtin_assume(steps >= 1);  // g < n: the group's first step always exists
      float pi[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) pi[u] = 0.f;
      auto block = [&](auto bc) {
        constexpr int b = decltype(bc)::value;
        constexpr int s0 = b * STEPS;
        if constexpr (b % 2 == 0) {
          if constexpr (b + 1 < NB) gather_block<DP, STEPS, AUG>(a1, r1, jv, rv, s0 + STEPS, Fp, aug_lane);
          mma_block<DP, STEPS, AUG>(acc, rhs, xo, pi, a0, r0, s0, steps);
        } else {
          if constexpr (b + 1 < NB) gather_block<DP, STEPS, AUG>(a0, r0, jv, rv, s0 + STEPS, Fp, aug_lane);
          else gather_block<DP, STEPS, AUG>(a0, r0, jn, rn, 0, Fp, aug_lane);
          mma_block<DP, STEPS, AUG>(acc, rhs, xo, pi, a1, r1, s0, steps);
        }
      };
      unroll_blocks<0, NB>(block);
      group_residuals(pi, rv, g, n, sse);
      jv = jn;
      rv = rn;
    }
  }
}

}  // namespace als
