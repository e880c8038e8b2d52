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

// Sum over the four row groups (lanes l, l ^ 16, l ^ 32, l ^ 48), in every lane: the
// 16-lane swap of a value with itself gives row groups {0, 0, 2, 2} and {1, 1, 3, 3},
// whose sum the 32-lane swap then pairs across the halves. The additions associate as
// (r0 + r1) + (r2 + r3), as the two butterfly steps xor 16 then xor 32 do, without the
// round trips through the LDS unit that those shuffles take.
__device__ __forceinline__ float sum_row_groups(float v) {
  const unsigned u = __float_as_uint(v);
  const auto h = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float s = __uint_as_float(h[0]) + __uint_as_float(h[1]);
  const unsigned t = __float_as_uint(s);
  const auto g = __builtin_amdgcn_permlane32_swap(t, t, false, false);
  return __uint_as_float(g[0]) + __uint_as_float(g[1]);
}

// Rotate a value right by K lanes within each 16-lane row (DPP row_ror).
template <int K>
__device__ __forceinline__ float row_ror(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x120 + K, 0xF, 0xF, false));
}

// Sum over the 16 lanes of a row; every lane of the row receives the same value.
// Sum of a double over the 64 lanes, in every lane: rotations within each 16-lane row
// (both 32-bit halves moved by DPP), then the two swaps across the row groups. A fixed
// order, so the result is the same on every run.
template <int K>
__device__ __forceinline__ double row_ror_f64(double v) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(v);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(unsigned)b, 0x120 + K, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(unsigned)(b >> 32), 0x120 + K, 0xF, 0xF, false);
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}
__device__ __forceinline__ double sum_wave_f64(double v) {
  v += row_ror_f64<8>(v);
  v += row_ror_f64<4>(v);
  v += row_ror_f64<2>(v);
  v += row_ror_f64<1>(v);
  const unsigned long long b = (unsigned long long)__double_as_longlong(v);
  const unsigned lo = (unsigned)b, hi = (unsigned)(b >> 32);
  auto join = [](unsigned l, unsigned h) {
    return __longlong_as_double((long long)(((unsigned long long)h << 32) | l));
  };
  const auto l16 = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
  const auto h16 = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
  const double s = join(l16[0], h16[0]) + join(l16[1], h16[1]);
  const unsigned long long bs = (unsigned long long)__double_as_longlong(s);
  const unsigned slo = (unsigned)bs, shi = (unsigned)(bs >> 32);
  const auto l32 = __builtin_amdgcn_permlane32_swap(slo, slo, false, false);
  const auto h32 = __builtin_amdgcn_permlane32_swap(shi, shi, false, false);
  return join(l32[0], h32[0]) + join(l32[1], h32[1]);
}

__device__ __forceinline__ float sum16(float v) {
  v += row_ror<8>(v);
  v += row_ror<4>(v);
  v += row_ror<2>(v);
  v += row_ror<1>(v);
  return v;
}

// Lane permutations within 16-lane rows (DPP): mirror within each half-row
// (lane i <-> 7 - i) and swaps within quads (lane i <-> i ^ 2, i <-> i ^ 1).
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppHalfMirror = 0x141, kDppQuadXor2 = 0x4E, kDppQuadXor1 = 0xB1;

// Four 16-lane row sums at once (reduce-scatter): afterwards lane c of a row holds
// the row's sum of s[c >> 2]. Partners at each level share every lane bit above the
// one that decides which half a lane keeps, so each lane ends with the full sum.
__device__ __forceinline__ float sum16x4(float s0, float s1, float s2, float s3) {
  const int c = threadIdx.x & 15;
  const bool h8 = (c & 8) != 0, h4 = (c & 4) != 0;
  const float k0 = h8 ? s2 : s0, k1 = h8 ? s3 : s1;  // kept half
  const float g0 = h8 ? s0 : s2, g1 = h8 ? s1 : s3;  // half given to lane c ^ 8
  const float t0 = k0 + row_ror<8>(g0), t1 = k1 + row_ror<8>(g1);
  float u = (h4 ? t1 : t0) + dpp_move<kDppHalfMirror>(h4 ? t0 : t1);
  u += dpp_move<kDppQuadXor2>(u);
  u += dpp_move<kDppQuadXor1>(u);
  return u;
}

// Value of lane (kq, c & 3), i.e. lane 16 kq + (c & 3): ds_swizzle in bit mode with and-mask
// 0x13 keeps lane bits 0, 1 and 4 within each 32-lane half.
__device__ __forceinline__ float from_row_lane03(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), 0x13));
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

// 1 / sqrt(p) without the clamp, for a factorisation that discards the whole system when
// a pivot is not positive and finite (the NaN or infinity it then produces stays in that
// system); two dependent instructions shorter per pivot.
__device__ __forceinline__ float inv_sqrt_pivot_raw(float p) { return __builtin_amdgcn_rsqf(p); }

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

// Per-wave LDS staging of a 64-rating group's column indices and ratings, transposed
// so that lane (kq, c) finds the values of its steps s (ratings 4 s + kq) contiguously
// at [kq * 16 + s]; two buffers let the next group be staged while the current one is
// still read.
struct GroupStage {
  int32_t j[2][64];
  float r[2][64];
  float w[2][64];   // per-rating weights (weighted ALS only)
  int32_t t[2][64]; // second index of each rating (tensor ALS only)
  // the 16 step partials of every lane, transposed for the end-of-group sums: row group kq,
  // feature lane c, step s at [kq * kRedGroup + c * kRedRow + s]; the odd row stride keeps
  // both the row-wise stores and the column-wise loads free of bank conflicts
  float red[4 * 16 * 17];
};
constexpr int kRedRow = 17, kRedGroup = 16 * kRedRow;

// One rating per lane of a 64-rating group: column index, rating, weight and (tensor
// ALS) the index into the second fixed table.
struct GroupLanes {
  int j;
  float r;
  float w;
  int t;
};

// Stage the group held one rating per lane (lane L holds rating L of the group).
template <bool WT, bool TS = false>
__device__ __forceinline__ void stage_group(GroupStage &st, int buf, const GroupLanes &g) {
  const int lane = threadIdx.x & 63;
  const int at = (lane & 3) * 16 + (lane >> 2);
  st.j[buf][at] = g.j;
  st.r[buf][at] = g.r;
  if constexpr (WT) st.w[buf][at] = g.w;
  if constexpr (TS) st.t[buf][at] = g.t;
}

// Rating `first + lane` of an item (n ratings): clamped loads, then the all-zero row,
// rating 0, weight 0 and second index 0 past the item's end.
template <bool WT, bool TS = false>
__device__ __forceinline__ GroupLanes group_lanes(const int32_t *__restrict__ ip,
                                                  const uint8_t *__restrict__ vp,
                                                  const float *__restrict__ wp,
                                                  const int32_t *__restrict__ tp, int n,
                                                  int first, int zrow) {
  const int k = first + (int)(threadIdx.x & 63);
  const int kc = min(k, n - 1);
  const int j = ip[kc];
  const float r = (float)vp[kc];
  GroupLanes g;
  g.j = k < n ? j : zrow;
  g.r = k < n ? r : 0.f;
  if constexpr (WT) {
    const float w = wp[kc];
    g.w = k < n ? w : 0.f;
  } else {
    g.w = 1.f;
  }
  if constexpr (TS) {
    const int t = tp[kc];
    g.t = k < n ? t : 0;
  } else {
    g.t = 0;
  }
  return g;
}

// The first group of an item (group_lanes(.., 0, ..)); an item without ratings gets the
// empty group (the all-zero row, rating 0, weight 0) and reads no rating.
template <bool WT, bool TS = false>
__device__ __forceinline__ GroupLanes first_group(const int32_t *__restrict__ ip,
                                                  const uint8_t *__restrict__ vp,
                                                  const float *__restrict__ wp,
                                                  const int32_t *__restrict__ tp, int n,
                                                  int zrow) {
  if (n <= 0) return GroupLanes{zrow, 0.f, 0.f, 0};
  return group_lanes<WT, TS>(ip, vp, wp, tp, n, 0, zrow);
}

// Gather the staged fixed rows of steps s0 .. s0 + STEPS - 1 of a 64-rating group:
// lane (kq, c) receives feature 16 X + c of rating 4 s + kq. The group's column
// indices and ratings come from its staging buffer.
// Loads are never predicated per lane (a predicated load becomes a branch that waits
// for its own completion, which serialises the gathers): ratings past the end of the
// item read the staged all-zero row, and padded features read the staged row's zero
// padding. One 32-bit byte offset per step from the (uniform) table base; the tiles
// follow at immediate offsets.
// With AUG, lane column aug_c of the last tile carries the rating instead of the
// (zero) padded feature, so that the MFMA Gram also accumulates b = sum r f in that
// column (and sum r^2 on its diagonal).
// With TS (tensor ALS) the fixed vector is the elementwise product of the rows of two
// staged tables, Fp[j] * Tp[t] (t the rating's second index); the padding of Fp keeps
// the product's padding zero.
// With STRIP, sb[u] receives feature 16 (T - 1) + (c & 3) of the lane's rating: the
// operand that every 4x4 block of the strip products in mma_block multiplies by.
template <int DP, int STEPS, bool AUG, bool WT, bool TS = false, bool STRIP = false>
__device__ __forceinline__ void gather_block(float (&a)[STEPS][DP / 16], float (&sb)[STEPS],
                                             float (&r)[STEPS], float (&wt)[STEPS],
                                             const GroupStage &st, int buf, int s0,
                                             const float *__restrict__ Fp,
                                             const float *__restrict__ Tp, bool aug_lane) {
  constexpr int T = DP / 16;
  const int lane = threadIdx.x & 63;
  const int kq = lane >> 4, c = lane & 15;
  const int32_t *__restrict__ sj = &st.j[buf][kq * 16 + s0];
  const float *__restrict__ sr = &st.r[buf][kq * 16 + s0];
  const float *__restrict__ sw = &st.w[buf][kq * 16 + s0];
  const int32_t *__restrict__ stt = &st.t[buf][kq * 16 + s0];
#pragma unroll
  for (int u = 0; u < STEPS; ++u) {
    const int j = sj[u];
    r[u] = sr[u];
    wt[u] = WT ? sw[u] : 1.f;
    const uint32_t off = (uint32_t)j * (uint32_t)(DP * 4) + (uint32_t)(c * 4);
    const char *row = reinterpret_cast<const char *>(Fp) + (uint64_t)off;
#pragma unroll
    for (int X = 0; X < T; ++X) a[u][X] = *reinterpret_cast<const float *>(row + 64 * X);
    // the strip operand sits 4 (c & 3) bytes into the last tile of the same row
    const int strip_off = 64 * (T - 1) - 4 * (c & 12);
    if constexpr (STRIP) sb[u] = *reinterpret_cast<const float *>(row + strip_off);
    if constexpr (TS) {
      const uint32_t off2 = (uint32_t)stt[u] * (uint32_t)(DP * 4) + (uint32_t)(c * 4);
      const char *row2 = reinterpret_cast<const char *>(Tp) + (uint64_t)off2;
#pragma unroll
      for (int X = 0; X < T; ++X) a[u][X] *= *reinterpret_cast<const float *>(row2 + 64 * X);
      if constexpr (STRIP) sb[u] *= *reinterpret_cast<const float *>(row2 + strip_off);
    }
    if constexpr (AUG) a[u][T - 1] = aug_lane ? r[u] : a[u][T - 1];
  }
}

// MFMA Gram update, right-hand side and per-step partial predictions of the gathered
// steps s0 .. s0 + STEPS - 1, in sub-blocks of up to four steps; sub-blocks past the
// item's last step (steps of this group) are skipped. With AUG the right-hand side is
// a column of the Gram and rhs is left alone. With WT (weighted ALS) the first MFMA
// operand carries c f, so the tiles accumulate sum c f f^T (and, in the augmented
// column, sum c r f); predictions use the unweighted rows.
// CORNER (two tiles, features 16..20 used in the second: the one-lane widths D = 17..20,
// always with STRIP): the last diagonal tile would spend a 16x16 MFMA on 15 useful
// products, so it is skipped. With CMFMA its 4 x 4 block of used features takes one
// v_mfma_f32_4x4x1f32 of the strip operand with itself into the tile's (otherwise unused)
// accumulator (each rating's four blocks agree; the caller keeps the first), and the
// right-hand side of features 16..19 accumulates in corner on VALU. Without CMFMA (tensor
// ALS, whose steps this extra MFMA slows) each lane c < 15 of a row group accumulates one
// product f[16 + p] f[16 + q] of the group's rating, fetching the two values across the
// group's lanes with ds_bpermute (byte addresses cx, cy) and adding them with one FMA.
// STRIP (only features 16 (T - 1) .. 16 (T - 1) + 3 used in the last tile): the tiles
// (I, T - 1) of the last column would spend a 16x16 MFMA each on four useful columns, so
// each takes one v_mfma_f32_4x4x1f32 instead. Its 16 blocks are b = 4 kq + cb: block b
// multiplies rows 16 I + 4 cb .. + 3 (the lane's own operand) by the four used features
// of the last tile (sb), for rating kq alone; acc[tidx(I, T - 1)] then holds these
// per-rating strips until strip_finish sums and rearranges them.
template <int DP, int STEPS, bool AUG, bool WT, bool CORNER = false, bool STRIP = false,
          bool CMFMA = false>
__device__ __forceinline__ void mma_block(floatx4 (&acc)[RowCfg<DP>::NT],
                                          float (&rhs)[DP / 16], const float (&xo)[DP / 16],
                                          float (&pi)[16], const float (&a)[STEPS][DP / 16],
                                          const float (&sb)[STEPS], const float (&r)[STEPS],
                                          const float (&wt)[STEPS], int s0, int steps,
                                          float &corner, int cx, int cy) {
  constexpr int T = DP / 16, SUB = STEPS < 4 ? STEPS : 4;
  static_assert(!CORNER || T == 2, "the corner path is for two tiles");
  static_assert(!STRIP || (T >= 3 && !AUG && !CORNER) || (T == 2 && AUG && CORNER),
                "the strip path is for three or more tiles with the right-hand side in rhs, or "
                "for the two-tile corner widths");
  // two-tile strip (with CORNER): the strip operand is feature 16 + (c & 3) of the lane's
  // rating, which lane c & 3 of the same row group holds in its second block; a swizzle
  // fetches it without a second load
  constexpr bool STRIP2 = STRIP && T == 2;
#pragma unroll
  for (int u0 = 0; u0 < STEPS; u0 += SUB) {
    if (s0 + u0 < steps) {
#pragma unroll
      for (int u = u0; u < u0 + SUB; ++u) {
        const float rw = WT ? wt[u] * r[u] : r[u];
        float wa[T];
#pragma unroll
        for (int X = 0; X < T; ++X) {
          wa[X] = WT ? wt[u] * a[u][X] : a[u][X];
          if constexpr (!AUG) rhs[X] = fmaf(rw, a[u][X], rhs[X]);
          pi[s0 + u] = fmaf(a[u][X], xo[X], pi[s0 + u]);
        }
        // the two-tile strip leaves the augmented column out: features 0..15 take their
        // right-hand side on VALU (16..19 take it in the corner products)
        if constexpr (STRIP2) rhs[0] = fmaf(rw, a[u][0], rhs[0]);
        const float sbu = STRIP2 ? from_row_lane03(a[u][T - 1]) : sb[u];
#pragma unroll
        for (int I = 0; I < T; ++I) {
#pragma unroll
          for (int J = I; J < T; ++J) {
            if (CORNER && I == T - 1) continue;
            if (STRIP && J == T - 1)
              acc[tidx<T>(I, J)] =
                  __builtin_amdgcn_mfma_f32_4x4x1f32(wa[I], sbu, acc[tidx<T>(I, J)], 0, 0, 0);
            else
              acc[tidx<T>(I, J)] = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[I], a[u][J],
                                                                        acc[tidx<T>(I, J)], 0, 0, 0);
          }
        }
        if constexpr (CORNER && CMFMA) {
          const float ws = WT ? wt[u] * sbu : sbu;
          acc[tidx<T>(T - 1, T - 1)] =
              __builtin_amdgcn_mfma_f32_4x4x1f32(ws, sbu, acc[tidx<T>(T - 1, T - 1)], 0, 0, 0);
          corner = fmaf(rw, sbu, corner);
        } else if constexpr (CORNER) {
          const float xv = __builtin_bit_cast(
              float, __builtin_amdgcn_ds_bpermute(cx, __builtin_bit_cast(int, wa[T - 1])));
          const float yv = __builtin_bit_cast(
              float, __builtin_amdgcn_ds_bpermute(cy, __builtin_bit_cast(int, a[u][T - 1])));
          corner = fmaf(xv, yv, corner);
        }
      }
    }
  }
}

// End of a 64-rating group: every lane stores its 16 step partials (feature lane c's
// share of the predictions of steps 0..15 of its rating group) to LDS, then lane (kq, c)
// sums the 16 feature lanes' shares of step c in lane order, which gives the full
// prediction of rating g + 4 c + kq; its squared residual is added to sse.
__device__ __forceinline__ void group_residuals(const float (&pi)[16], GroupStage &st, int buf,
                                                int g, int n, double &sse) {
  const int lane = threadIdx.x & 63;
  const int kq = lane >> 4, c = lane & 15;
  float *row = &st.red[kq * kRedGroup + c * kRedRow];
#pragma unroll
  for (int u = 0; u < 16; ++u) row[u] = pi[u];
  wave_sync();
  const float *col = &st.red[kq * kRedGroup + c];
  float p = col[0];
#pragma unroll
  for (int q = 1; q < 16; ++q) p += col[q * kRedRow];
  const float rq = st.r[buf][kq * 16 + c];
  wave_sync();  // the area is rewritten by the next group
  if (g + 4 * c + kq < n) {
    const double e = (double)rq - (double)p;
    sse = fma(e, e, sse);
  }
}

// Accumulate the item's Gram tiles and right-hand side and the entering-state squared
// residuals. Without AUG the right-hand side is kept in rhs as per-lane partials over
// the four rating groups; with AUG it is the Gram's column 16 (T - 1) + aug_c (a padding
// column whose lane carries the ratings) and rhs is untouched.
// xo: the row's current factor values in lane-column form (xo[X] = x[16X + c]).
// wp: the item's per-rating weights (weighted ALS, WT), else unused.
// gv: the first group's lanes (group_lanes(.., 0, ..)), loaded by the caller.
// Ratings are taken in groups of 64, each gathered in blocks of STEPS steps (four
// ratings per step).
//  - Narrow rows (T <= 2): one block per group, gathered and then multiplied.
//  - Wider rows: two block buffers; the gather of the next block (of this group, or
//    the first block of the next group) is issued before the MFMAs of the current
//    one, so that its latency hides behind them. The blocks of the last group that
//    lie past the item's end are still gathered (from the zero row) but not multiplied.
// tp, Tp (tensor ALS, TS): the item's second indices and the second staged table.
// corner, cx, cy: the corner products of mma_block (CORNER; with CMFMA, for all but TS,
// only the right-hand side of features 16..19), else unused.
// STRIP: the last tile column in strip form (mma_block); the caller finishes it with
// strip_finish.
template <int DP, bool AUG, bool WT, bool TS = false, bool CORNER = false, bool STRIP = false>
__device__ __forceinline__ void gram_accumulate(floatx4 (&acc)[RowCfg<DP>::NT],
                                                float (&rhs)[RowCfg<DP>::T],
                                                const float (&xo)[RowCfg<DP>::T], double &sse,
                                                const int32_t *__restrict__ ip,
                                                const uint8_t *__restrict__ vp,
                                                const float *__restrict__ wp,
                                                const int32_t *__restrict__ tp, int n,
                                                const float *__restrict__ Fp,
                                                const float *__restrict__ Tp, int zrow,
                                                int aug_c, GroupStage &st, GroupLanes gv,
                                                float &corner, int cx, int cy) {
  using C = RowCfg<DP>;
  constexpr int T = C::T, STEPS = C::STEPS, NB = 16 / STEPS;
  const int lane = threadIdx.x & 63;
  const bool aug_lane = (lane & 15) == aug_c;
  if constexpr (T <= 2) {
    for (int g = 0; g < n; g += 64) {
      const GroupLanes gn = group_lanes<WT, TS>(ip, vp, wp, tp, n, g + 64, zrow);
      const int steps = min(16, (n - g + 3) >> 2);
      __builtin_assume(steps >= 1);  // g < n: the group's first step always exists
      stage_group<WT, TS>(st, 0, gv);
      wave_sync();
      float pi[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) pi[u] = 0.f;
#pragma unroll
      for (int s0 = 0; s0 < 16; s0 += STEPS) {
        if (s0 < steps) {
          float a[STEPS][T];
          float sb[STEPS], r[STEPS], w[STEPS];
          gather_block<DP, STEPS, AUG, WT, TS>(a, sb, r, w, st, 0, s0, Fp, Tp, aug_lane);
          mma_block<DP, STEPS, AUG, WT, CORNER, STRIP, CORNER && !TS>(acc, rhs, xo, pi, a, sb, r, w, s0, steps,
                                                       corner, cx, cy);
        }
      }
      group_residuals(pi, st, 0, g, n, sse);
      wave_sync();  // the buffer is restaged by the next group
      gv = gn;
    }
  } else {
    static_assert(NB % 2 == 0, "block buffers alternate within and across groups");
    float a0[STEPS][T], a1[STEPS][T], b0[STEPS], b1[STEPS], r0[STEPS], r1[STEPS], w0[STEPS],
        w1[STEPS];
    stage_group<WT, TS>(st, 0, gv);
    wave_sync();
    gather_block<DP, STEPS, AUG, WT, TS, STRIP>(a0, b0, r0, w0, st, 0, 0, Fp, Tp, aug_lane);
    int buf = 0;
    for (int g = 0; g < n; g += 64) {
      const GroupLanes gn = group_lanes<WT, TS>(ip, vp, wp, tp, n, g + 64, zrow);
      const int steps = min(16, (n - g + 3) >> 2);
      __builtin_assume(steps >= 1);  // g < n: the group's first step always exists
      float pi[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) pi[u] = 0.f;
      auto block = [&](auto bc) {
        constexpr int b = decltype(bc)::value;
        constexpr int s0 = b * STEPS;
        if constexpr (b % 2 == 0) {
          if constexpr (b + 1 < NB)
            gather_block<DP, STEPS, AUG, WT, TS, STRIP>(a1, b1, r1, w1, st, buf, s0 + STEPS, Fp,
                                                        Tp, aug_lane);
          mma_block<DP, STEPS, AUG, WT, CORNER, STRIP, CORNER && !TS>(acc, rhs, xo, pi, a0, b0, r0, w0, s0,
                                                       steps, corner, cx, cy);
        } else {
          if constexpr (b + 1 < NB) {
            gather_block<DP, STEPS, AUG, WT, TS, STRIP>(a0, b0, r0, w0, st, buf, s0 + STEPS, Fp,
                                                        Tp, aug_lane);
          } else {
            // the next group goes to the other buffer, then its first block is gathered
            stage_group<WT, TS>(st, buf ^ 1, gn);
            wave_sync();
            gather_block<DP, STEPS, AUG, WT, TS, STRIP>(a0, b0, r0, w0, st, buf ^ 1, 0, Fp, Tp,
                                                        aug_lane);
          }
          mma_block<DP, STEPS, AUG, WT, CORNER, STRIP, CORNER && !TS>(acc, rhs, xo, pi, a1, b1, r1, w1, s0,
                                                       steps, corner, cx, cy);
        }
      };
      unroll_blocks<0, NB>(block);
      group_residuals(pi, st, buf, g, n, sse);
      buf ^= 1;
    }
  }
}

// Whether the last tile of width DP uses only its first four features (D in
// 16 (T - 1) + 1 .. 16 (T - 1) + 4, three to seven tiles): then the strip form of
// mma_block serves the last tile column, and the augmented column is feature
// 16 (T - 1) + 4. At eight tiles the strip form spills several times more registers
// than the tile form, so those widths keep the tile form.
template <int DP>
__host__ __device__ constexpr bool strip_width(int D) {
  return DP / 16 >= 3 && DP / 16 <= 7 && D > DP - 16 && D <= DP - 12;
}

// Finish a strip-form Gram (mma_block with STRIP): sum each strip of the last tile
// column over the four rating groups and move it to the tile layout (lane (kq, c), c < 4,
// element r: G[16 I + 4 kq + r][16 (T - 1) + c], taken from lane 4 kq + c of the summed
// strip), and write the right-hand side (per-lane partials in rhs) into lane column aug_c
// of the same tiles (element r: b[16 I + 4 kq + r], from lane 4 kq + r of the summed rhs).
// The other lane columns of these tiles become zero. (Here the row-group sums stay LDS
// shuffles: with seven or eight tiles their latency overlaps, and the lane swaps of
// sum_row_groups measured slower.)
template <int DP>
__device__ __forceinline__ void strip_finish(floatx4 (&acc)[RowCfg<DP>::NT],
                                             float (&rhs)[DP / 16], int aug_c) {
  constexpr int T = DP / 16;
  const int lane = threadIdx.x & 63, kq = lane >> 4, c = lane & 15;
  const int from_strip = 4 * (4 * kq + (c & 3));
#pragma unroll
  for (int I = 0; I < T; ++I) {
    floatx4 s = acc[tidx<T>(I, T - 1)];
    float b = rhs[I];
    b += __shfl_xor(b, 16);
    b += __shfl_xor(b, 32);
    floatx4 out;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v = s[r];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      const float sv = __builtin_bit_cast(
          float, __builtin_amdgcn_ds_bpermute(from_strip, __builtin_bit_cast(int, v)));
      const float bv = __builtin_bit_cast(
          float, __builtin_amdgcn_ds_bpermute(4 * (4 * kq + r), __builtin_bit_cast(int, b)));
      out[r] = c < 4 ? sv : (c == aug_c ? bv : 0.f);
    }
    acc[tidx<T>(I, T - 1)] = out;
  }
}

}  // namespace als
