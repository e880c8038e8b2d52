// The fused row kernel of the ALS half-sweep (Sec. 2.2): for each row s of the
// solved side, one wavefront
//   1. accumulates the normal equations G = sum_k f_k f_k^T (upper-triangle
//      16x16 tiles, fp32 MFMA 16x16x4, held in accumulator registers) and
//      b = sum_k r_k f_k over the row's ratings, and on the same gathered rows
//      the squared residuals (r_k - x_s . f_k)^2 of the state entering the
//      half-sweep (x_s = the row's previous value) for the training RMSE
//      (Sec. 4.1);
//   2. factors A = U^T U (lambda n_s I is the accumulators' initial value) in
//      panels of four rows: the 4x4 diagonal block is factored in every lane and
//      inverted (M = U_gg^{-T}), each lane forms its panel row of U with one
//      4-term dot product per tile, and the trailing tiles are updated on MFMA
//      (K = 4). The accumulators are only written by MFMA and read by VALU;
//   3. forward substitution of b rides along the panels (as a column of the
//      matrix when a padding feature can carry it); back substitution follows,
//      from the untouched panel rows A_p and the stored M blocks; x_s is written
//      unless a pivot was not positive and finite.
// Rows with more ratings than the hub threshold have their normal equations
// built by several wavefronts (k_gram_chunks, partials in a workspace) and are
// only summed and solved here.
// STRIP (the last tile holds four used features, D = 16 (T - 1) + 1 .. + 4): the
// Gram's last tile column is accumulated as 4x4 strips (v_mfma_f32_4x4x1f32) and the
// right-hand side on VALU, and both are moved into the augmented tile layout before
// the factorisation, which is the same as without STRIP.
//
// Register layout: lane (kq, c) = (lane / 16, lane % 16). Gram operand block X
// of rating k is feature 16 X + c of f_k in lane (k, c). Accumulator tile
// (I, J), I <= J, holds A[16 I + 4 kq + r][16 J + c] in element r. The fixed
// side is read from a staged copy with row stride DP (zero padded), so every
// gathered row starts on a 64-byte boundary.
#include "gram.h"

namespace als {

// Copy the fixed factors [n x D] into a zero-padded [(n + 1) x DP] buffer whose
// last row is all zero (the stand-in of absent ratings). Thread (q, y) of a block
// writes float4 q of staged row blockIdx.x * blockDim.y + y (grid-stride over rows).
__global__ void k_stage_fixed(const float *__restrict__ F, int64_t n, int D, int DP,
                              float *__restrict__ Fp) {
  const int q = threadIdx.x;
  const int d0 = 4 * q;
  for (int64_t row = (int64_t)blockIdx.x * blockDim.y + threadIdx.y; row <= n;
       row += (int64_t)gridDim.x * blockDim.y) {
    float v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = (row < n && d0 + k < D) ? F[row * D + d0 + k] : 0.f;
    *reinterpret_cast<float4 *>(Fp + row * DP + d0) = make_float4(v[0], v[1], v[2], v[3]);
  }
}

hipError_t launch_stage_fixed(const float *F, int64_t n, int D, int DP, float *Fp, hipStream_t s) {
  if (n < 0 || DP % 4 != 0 || DP / 4 > 256) return hipErrorInvalidValue;
  const int dp4 = DP / 4;
  const int rows_per_block = 256 / dp4;
  int64_t blocks = (n + 1 + rows_per_block - 1) / rows_per_block;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_stage_fixed, dim3((unsigned)blocks), dim3(dp4, rows_per_block), 0, s, F, n,
                     D, DP, Fp);
  return hipGetLastError();
}

// The augmented column: when DA = 4 ceil(D / 4) is a padding feature (DA < DP), the
// gathered rows carry the rating in feature DA, so the Gram's column DA is b = sum r f
// and the elimination of A = U^T U carries b along as y = U^{-T} b. DA always falls in
// the last tile; aug_c is its lane column there.
template <int DP>
__host__ __device__ constexpr int aug_column(int D) {
  return ((D + 3) & ~3) - 16 * (DP / 16 - 1);
}

// Partial normal equations of the chunks of split rows, with the chunks'
// entering-state squared residuals.
template <int DP, bool AUG, bool WT, bool TS, bool STRIP = false>
__global__ __launch_bounds__(64) void k_gram_chunks(const WorkItem *__restrict__ items,
                                                    const int32_t *__restrict__ idx,
                                                    const uint8_t *__restrict__ val,
                                                    const float *__restrict__ wts,
                                                    const float *__restrict__ Fp, int zrow,
                                                    const float *__restrict__ Xold, int D,
                                                    float *__restrict__ ws,
                                                    double *__restrict__ sse_out, Hadamard hd) {
  using C = RowCfg<DP>;
  constexpr int T = C::T, NT = C::NT;
  __shared__ GroupStage s_stage;
  const WorkItem it = items[blockIdx.x];
  const int lane = threadIdx.x, kq = lane >> 4, c = lane & 15;
  floatx4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  float rhs[T], xo[T];
#pragma unroll
  for (int X = 0; X < T; ++X) {
    rhs[X] = 0.f;
    {
      const float v = Xold[(int64_t)it.row * D + min(16 * X + c, D - 1)];
      xo[X] = 16 * X + c < D ? v : 0.f;
    }
  }
  double sse = 0.0;
  const float *__restrict__ wp = WT ? wts + it.start : nullptr;
  const int32_t *__restrict__ tp = TS ? hd.idx2 + it.start : nullptr;
  const GroupLanes g0 =
      first_group<WT, TS>(idx + it.start, val + it.start, wp, tp, it.len, zrow);
  float no_corner = 0.f;
  const int aug_c = AUG ? aug_column<DP>(D) : -1;
  gram_accumulate<DP, AUG && !STRIP, WT, TS, false, STRIP>(
      acc, rhs, xo, sse, idx + it.start, val + it.start, wp, tp, it.len, Fp, hd.Tp, zrow,
      STRIP ? -1 : aug_c, s_stage, g0, no_corner, 0, 0);
  if constexpr (STRIP) strip_finish<DP>(acc, rhs, aug_c);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sse += __shfl_xor(sse, o);
  float *__restrict__ out = ws + it.slot * (int64_t)slot_floats(DP);
#pragma unroll
  for (int t = 0; t < NT; ++t) *reinterpret_cast<floatx4 *>(out + t * 256 + lane * 4) = acc[t];
  if constexpr (!AUG) {
#pragma unroll
    for (int X = 0; X < T; ++X) {
      rhs[X] += __shfl_xor(rhs[X], 16);
      rhs[X] += __shfl_xor(rhs[X], 32);
    }
    if (kq == 0) {
#pragma unroll
      for (int X = 0; X < T; ++X) out[NT * 256 + 16 * X + c] = rhs[X];
    }
  }
  if (lane == 0) sse_out[blockIdx.x] = sse;
}

constexpr int kRowWaves = 1;  // rows per workgroup (one per wavefront)

// Two wavefronts per SIMD (the second launch bound) outweigh the few registers the
// wide widths then spill: the accumulator tiles move to arch VGPRs and the gather
// latency of one row hides behind the other row's MFMAs.
//
// Panel step (rows p0 .. p0 + 3, held by row group g of tile row I0):
//   the 4x4 diagonal block A_gg = U_gg^T U_gg is factored in every lane and
//   M = U_gg^{-T} formed explicitly (10 entries); lane (kq, c) then forms the panel
//   row U[p0 + kq][j] = sum_r M[kq][r] A[p0 + r][j] for its columns j = 16 X + c
//   with one 4-term dot product per tile, and the trailing tiles are updated on MFMA
//   (K = 4). Without the augmented column the right-hand side is eliminated along:
//   y_p = M b_p, and b_j -= sum_r A[p0 + r][j] (M^T y_p)_r for the later columns.
//
// BAYES (a Gibbs half-sweep): the accumulators start from the prior image (Lambda /
// alpha, identity on the padding, and Lambda mu / alpha in the right-hand side) and the
// forward-substitution result y gets z / sqrt(alpha) before the back substitution, so
// that the row receives the conditional draw mu* + L*^{-T} z. For the time chain of BPTF
// the image is scaled per row and a per-row right-hand side h0 is added (RowPrior).
template <int DP, bool AUG, bool WT, bool BAYES, bool TS, bool STRIP = false>
__global__ __launch_bounds__(64 * kRowWaves, 2) void k_rows(
    const RowTask *__restrict__ rows, int64_t n_rows, const int32_t *__restrict__ idx,
    const uint8_t *__restrict__ val, const float *__restrict__ wts,
    const float *__restrict__ Fp, int zrow,
    const float *__restrict__ ws, int D, float lam, float *__restrict__ X_io,
    double *__restrict__ sse_out,
    int32_t *__restrict__ flag_count, double *__restrict__ cyc_gram,
    double *__restrict__ cyc_solve, RowPrior pr, Hadamard hd) {
  const uint64_t t_start = __builtin_readcyclecounter();
  using C = RowCfg<DP>;
  constexpr int T = C::T, NT = C::NT;
  constexpr int NPAN = DP / 4;
  // tile row I0 of the panel step, as published by each row group: [row group][tile column][lane column]
  __shared__ floatx4 s_panel[kRowWaves][4][T][16];
  // per panel: M as a full 4 x 4 row-major block (zeros above the diagonal), then y_p
  __shared__ __attribute__((aligned(16))) float s_ud[kRowWaves][NPAN][20];
  __shared__ float s_dummy[kRowWaves][64];  // sink of the stores of lanes without an entry
  __shared__ GroupStage s_stage[kRowWaves];        // gather staging of the row's rating groups

  const int wv = threadIdx.x >> 6;
  const int64_t task = (int64_t)blockIdx.x * kRowWaves + wv;
  if (task >= n_rows) return;
  const RowTask rt = rows[task];
  const int lane = threadIdx.x & 63, kq = lane >> 4, c = lane & 15;
  floatx4(&panel)[4][T][16] = s_panel[wv];
  float(&ud)[NPAN][20] = s_ud[wv];
  float(&dummy)[64] = s_dummy[wv];
  const int aug_c = AUG ? aug_column<DP>(D) : -1;

  // A starts as lambda n_s I on the first D diagonal entries and I on the padding (only
  // the last tile holds padding); the Gram (or the sum of a split row's chunk partials)
  // is accumulated on top. With STRIP the last tile column starts from zero (it holds
  // strips during the Gram) and receives its initial value afterwards.
  const float lam_n = (float)((double)lam * (double)rt.deg);
  const float pscale = BAYES ? pr.scale_of(rt.row) : 1.f;
  auto tile_init = [&](int I, int J) -> floatx4 {
    if constexpr (BAYES) {
      return pscale *
             *reinterpret_cast<const floatx4 *>(pr.init + tidx<T>(I, J) * 256 + lane * 4);
    } else {
      floatx4 v = floatx4{0.f, 0.f, 0.f, 0.f};
      if (I == J) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int d = 16 * I + 4 * kq + r;
          v[r] = c == 4 * kq + r ? ((I < T - 1 || d < D) ? lam_n : 1.f) : 0.f;
        }
      }
      return v;
    }
  };
  floatx4 acc[NT];
#pragma unroll
  for (int I = 0; I < T; ++I) {
#pragma unroll
    for (int J = I; J < T; ++J)
      acc[tidx<T>(I, J)] = (STRIP && J == T - 1) ? floatx4{0.f, 0.f, 0.f, 0.f} : tile_init(I, J);
  }
  float rhs[T];
#pragma unroll
  for (int X = 0; X < T; ++X) rhs[X] = 0.f;

  float *__restrict__ xrow = X_io + (int64_t)rt.row * D;
  if (rt.nslots == 0) {
    float xo[T];
#pragma unroll
    for (int X = 0; X < T; ++X) {
      const float v = xrow[min(16 * X + c, D - 1)];
      xo[X] = 16 * X + c < D ? v : 0.f;
    }
    double sse = 0.0;
    const float *__restrict__ wp = WT ? wts + rt.start : nullptr;
    const int32_t *__restrict__ tp = TS ? hd.idx2 + rt.start : nullptr;
    const GroupLanes g0 =
        first_group<WT, TS>(idx + rt.start, val + rt.start, wp, tp, rt.deg, zrow);
    float no_corner = 0.f;
    gram_accumulate<DP, AUG && !STRIP, WT, TS, false, STRIP>(
        acc, rhs, xo, sse, idx + rt.start, val + rt.start, wp, tp, rt.deg, Fp, hd.Tp, zrow,
        STRIP ? -1 : aug_c, s_stage[wv], g0, no_corner, 0, 0);
    if constexpr (STRIP) strip_finish<DP>(acc, rhs, aug_c);
    if constexpr (!AUG) {
#pragma unroll
      for (int X = 0; X < T; ++X) {
        rhs[X] += __shfl_xor(rhs[X], 16);
        rhs[X] += __shfl_xor(rhs[X], 32);
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) sse += __shfl_xor(sse, o);
    if (lane == 0 && rt.sse_idx >= 0) sse_out[rt.sse_idx] = sse;
  } else {
    const float *__restrict__ base = ws + rt.slot0 * (int64_t)slot_floats(DP);
    for (int s = 0; s < rt.nslots; ++s) {
      const float *__restrict__ sl = base + s * (int64_t)slot_floats(DP);
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[t] += *reinterpret_cast<const floatx4 *>(sl + t * 256 + lane * 4);
      if constexpr (!AUG) {
#pragma unroll
        for (int X = 0; X < T; ++X) rhs[X] += sl[NT * 256 + 16 * X + c];
      }
    }
  }
  if constexpr (STRIP) {
#pragma unroll
    for (int I = 0; I < T; ++I) acc[tidx<T>(I, T - 1)] += tile_init(I, T - 1);
  }
  if constexpr (BAYES && !AUG) {
    // the prior's right-hand side (with the augmented column it sits in the tiles)
#pragma unroll
    for (int X = 0; X < T; ++X) rhs[X] = fmaf(pscale, pr.init[NT * 256 + 16 * X + c], rhs[X]);
  }
  if constexpr (BAYES) {
    // the time chain's per-row right-hand side: into the augmented column (every row group
    // holds its own rows there) or into rhs (every lane holds the full sums)
    if (pr.h0 != nullptr) {
      const float *__restrict__ hr = pr.h0 + (int64_t)rt.row * D;
      if constexpr (AUG) {
        if (c == aug_c) {
#pragma unroll
          for (int I = 0; I < T; ++I) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int d = 16 * I + 4 * kq + r;
              if (d < D) acc[tidx<T>(I, T - 1)][r] += hr[d];
            }
          }
        }
      } else {
#pragma unroll
        for (int X = 0; X < T; ++X)
          if (16 * X + c < D) rhs[X] += hr[16 * X + c];
      }
    }
  }

  const uint64_t t_gram = __builtin_readcyclecounter();

  // ---- factorisation A = U^T U with forward substitution U^T y = b ------------------------
  // Panel step (I0, g) of rows p0 .. p0 + 3, p0 = 16 I0 + 4 g. Its update of the trailing
  // tiles is split in two: the tiles that the next panel reads (tile row I0 while g < 3,
  // else tile row I0 + 1) are updated at once; the tiles below them are updated during
  // the next panel's step, in the same instruction stream as that step's dependent chain
  // of scalar-like work (diagonal block, pivots, M), so that the matrix unit runs while
  // the chain waits on its own latencies. The per-tile order of the updates is unchanged.
  bool bad = false;
  float up[T];  // the previous panel's rows U_p(:, 16 X + c) (its deferred update)
#pragma unroll
  for (int X = 0; X < T; ++X) up[X] = 0.f;
  // DEFER: the step issues its predecessor's deferred update; LAST: the step is the last
  // panel of its tile row (g = 3), whose immediate update is of tile row I0 + 1.
  // one-hot row-group selectors: lane (kq, c) takes row kq of M
  const float e0 = kq == 0 ? 1.f : 0.f, e1 = kq == 1 ? 1.f : 0.f;
  const float e2 = kq == 2 ? 1.f : 0.f, e3 = kq == 3 ? 1.f : 0.f;
  // and lane column c's entry of a row of M (the stores of step (5); zero past c = 3)
  const float f0 = c == 0 ? 1.f : 0.f, f1 = c == 1 ? 1.f : 0.f;
  const float f2 = c == 2 ? 1.f : 0.f, f3 = c == 3 ? 1.f : 0.f;
  auto panel_step = [&](auto i0c, auto deferc, auto lastc, int g) {
    constexpr int I0 = decltype(i0c)::value;
    constexpr bool DEFER = decltype(deferc)::value != 0;
    constexpr bool LAST = decltype(lastc)::value != 0;
    const int p0 = 16 * I0 + 4 * g;
    const int pan = p0 >> 2;
    // (0) the previous panel's update of the tiles below tile row I0
    if constexpr (DEFER) {
#pragma unroll
      for (int I = I0 + 1; I < T; ++I) {
#pragma unroll
        for (int J = I; J < T; ++J)
          acc[tidx<T>(I, J)] =
              __builtin_amdgcn_mfma_f32_16x16x4f32(-up[I], up[J], acc[tidx<T>(I, J)], 0, 0, 0);
      }
    }
    // (1) the 4x4 diagonal block A[p0 + r][p0 + r'] sits in element r of lane
    // (g, 4 g + r') of tile (I0, I0) and goes to scalar registers; every row group
    // publishes its rows of tile row I0 to LDS, and every lane reads row group g's
    // (the panel rows p0 .. p0 + 3) for its column
    const floatx4 dg = acc[tidx<T>(I0, I0)];
    const int l0 = 20 * g;
    const float a00 = lane_value(dg[0], l0), a01 = lane_value(dg[0], l0 + 1);
    const float a02 = lane_value(dg[0], l0 + 2), a03 = lane_value(dg[0], l0 + 3);
    const float a11 = lane_value(dg[1], l0 + 1), a12 = lane_value(dg[1], l0 + 2);
    const float a13 = lane_value(dg[1], l0 + 3), a22 = lane_value(dg[2], l0 + 2);
    const float a23 = lane_value(dg[2], l0 + 3), a33 = lane_value(dg[3], l0 + 3);
#pragma unroll
    for (int X = I0; X < T; ++X) panel[kq][X][c] = acc[tidx<T>(I0, X)];
    floatx4 col[T];
#pragma unroll
    for (int X = I0; X < T; ++X) col[X] = panel[g][X][c];
    // (2) 4x4 diagonal block, factored redundantly in every lane
    float p;
    p = a00;
    bad |= !(p > 0.f && p < INFINITY);
    const float i00 = inv_sqrt_pivot_raw(p);
    const float u01 = a01 * i00, u02 = a02 * i00, u03 = a03 * i00;
    p = a11 - u01 * u01;
    bad |= !(p > 0.f && p < INFINITY);
    const float i11 = inv_sqrt_pivot_raw(p);
    const float u12 = (a12 - u01 * u02) * i11, u13 = (a13 - u01 * u03) * i11;
    p = a22 - u02 * u02 - u12 * u12;
    bad |= !(p > 0.f && p < INFINITY);
    const float i22 = inv_sqrt_pivot_raw(p);
    const float u23 = (a23 - u02 * u03 - u12 * u13) * i22;
    p = a33 - u03 * u03 - u13 * u13 - u23 * u23;
    bad |= !(p > 0.f && p < INFINITY);
    const float i33 = inv_sqrt_pivot_raw(p);
    // M = U_gg^{-T} (lower triangular; diagonal 1 / u_qq)
    const float m00 = i00;
    const float m10 = -(u01 * m00) * i11, m11 = i11;
    const float m20 = -(u02 * m00 + u12 * m10) * i22, m21 = -(u12 * m11) * i22, m22 = i22;
    const float m30 = -(u03 * m00 + u13 * m10 + u23 * m20) * i33;
    const float m31 = -(u13 * m11 + u23 * m21) * i33, m32 = -(u23 * m22) * i33, m33 = i33;
    // this lane's row of M (row group kq holds panel row p0 + kq). With the augmented
    // column nothing else needs M as uniform values: row kq of U_gg^{-T} is column kq of
    // U_gg^{-1}, the back substitution of U_gg w = e_kq, ten instructions per lane instead
    // of M's sixteen and the selection's ten. Otherwise (y and v below need M) the row is
    // picked by one-hot sums, exact since every other term is a zero product; per-lane
    // selects of the uniform values compile to branches that sink the M terms into
    // divergent code.
    float w0, w1, w2, w3;
    if constexpr (AUG) {
      w3 = e3 * i33;
      w2 = (e2 - u23 * w3) * i22;
      w1 = (e1 - u12 * w2 - u13 * w3) * i11;
      w0 = (e0 - u01 * w1 - u02 * w2 - u03 * w3) * i00;
    } else {
      w0 = e0 * m00 + e1 * m10 + e2 * m20 + e3 * m30;
      w1 = e1 * m11 + e2 * m21 + e3 * m31;
      w2 = e2 * m22 + e3 * m32;
      w3 = e3 * m33;
    }
    float y0 = 0.f, y1 = 0.f, y2 = 0.f, y3 = 0.f;
    float v0 = 0.f, v1 = 0.f, v2 = 0.f, v3 = 0.f;
    if constexpr (!AUG) {
      // y_p = M b_p, and the weights v = M^T y_p of the right-hand-side update
      const float b0 = lane_value(rhs[I0], 4 * g + 0), b1 = lane_value(rhs[I0], 4 * g + 1);
      const float b2 = lane_value(rhs[I0], 4 * g + 2), b3 = lane_value(rhs[I0], 4 * g + 3);
      y0 = m00 * b0;
      y1 = m10 * b0 + m11 * b1;
      y2 = m20 * b0 + m21 * b1 + m22 * b2;
      y3 = m30 * b0 + m31 * b1 + m32 * b2 + m33 * b3;
      v0 = m00 * y0 + m10 * y1 + m20 * y2 + m30 * y3;
      v1 = m11 * y1 + m21 * y2 + m31 * y3;
      v2 = m22 * y2 + m32 * y3;
      v3 = m33 * y3;
    }
    // (3) panel rows U[p0 + kq][j] = (M A_p)[kq][j] for the later columns j (zero for
    // j <= p0 + 3, which keeps the finished rows and columns out of the update)
    float u[T];
#pragma unroll
    for (int X = 0; X < T; ++X) {
      u[X] = 0.f;
      if (X >= I0) {
        float Y = w0 * col[X][0];
        Y = fmaf(w1, col[X][1], Y);
        Y = fmaf(w2, col[X][2], Y);
        Y = fmaf(w3, col[X][3], Y);
        const int j = 16 * X + c;
        if (X == I0) Y = j > p0 + 3 ? Y : 0.f;
        if constexpr (!AUG) {
          if (j > p0 + 3)
            rhs[X] -= v0 * col[X][0] + v1 * col[X][1] + v2 * col[X][2] + v3 * col[X][3];
        }
        u[X] = Y;
      }
    }
    // (4) the update of the tiles that the next panel reads
    if constexpr (!LAST) {
#pragma unroll
      for (int J = I0; J < T; ++J)
        acc[tidx<T>(I0, J)] =
            __builtin_amdgcn_mfma_f32_16x16x4f32(-u[I0], u[J], acc[tidx<T>(I0, J)], 0, 0, 0);
    } else if constexpr (I0 + 1 < T) {
#pragma unroll
      for (int J = I0 + 1; J < T; ++J)
        acc[tidx<T>(I0 + 1, J)] = __builtin_amdgcn_mfma_f32_16x16x4f32(
            -u[I0 + 1], u[J], acc[tidx<T>(I0 + 1, J)], 0, 0, 0);
    }
#pragma unroll
    for (int X = 0; X < T; ++X) up[X] = u[X];
    // (5) M (row-major 4 x 4, zeros above the diagonal) and y_p for the back substitution.
    // Every lane stores, the lanes without an entry to a per-lane dummy slot: with
    // predicated stores each step would end a basic block, and the scheduler could not
    // interleave one step with the next.
    {
      const float wc = f0 * w0 + f1 * w1 + f2 * w2 + f3 * w3;
      *(c < 4 ? &ud[pan][4 * kq + c] : &dummy[lane]) = wc;
      if constexpr (AUG) {
        // the augmented column's panel entries are y_p = U_gg^{-T} b_p
        *(c == aug_c ? &ud[pan][16 + kq] : &dummy[lane]) = u[T - 1];
      } else {
        const float yc = f0 * y0 + f1 * y1 + f2 * y2 + f3 * y3;
        *(lane < 4 ? &ud[pan][16 + c] : &dummy[lane]) = yc;
      }
    }
  };
  // Rows from D on are padding: the steps stop at the first panel past D, and the updates
  // still deferred then only touch padding rows, which nothing reads.
  // D > 16 (T - 1), so every panel of the tile rows before the last is inside D and only
  // the last tile row needs the bound; without it the steps of the other tile rows form
  // one straight-line block that the scheduler can interleave across steps
  auto tile_row = [&](auto i0c) {
    constexpr int I0 = decltype(i0c)::value;
    // (the variants with an explicit right-hand side keep every bound: their longer
    // straight-line block spills)
    constexpr bool LASTROW = I0 == T - 1 || !AUG;
    // the first panel has no predecessor
    panel_step(i0c, IntC<I0 == 0 ? 0 : 1>{}, IntC<0>{}, 0);
    if (LASTROW && 16 * I0 + 4 >= D) return;
    panel_step(i0c, IntC<1>{}, IntC<0>{}, 1);
    if (LASTROW && 16 * I0 + 8 >= D) return;
    panel_step(i0c, IntC<1>{}, IntC<0>{}, 2);
    if (LASTROW && 16 * I0 + 12 >= D) return;
    panel_step(i0c, IntC<1>{}, IntC<1>{}, 3);
  };
  unroll_blocks<0, T>(tile_row);
  wave_sync();

  if constexpr (BAYES) {
    // y += z / sqrt(alpha): the panels keep y_p in ud[p][16 .. 19]
    const float *__restrict__ zr = pr.z + (int64_t)rt.row * D;
#pragma unroll
    for (int d0 = 0; d0 < DP; d0 += 64) {
      const int d = d0 + lane;
      if (d < D) ud[d >> 2][16 + (d & 3)] += pr.zscale * zr[d];
    }
    wave_sync();
  }

  // ---- back substitution U x = y --------------------------------------------------------
  // Panel p: U_gg x_p = y_p - U_p,rest x_rest with U_p,rest = M A_p,rest, where the
  // accumulators still hold the panel rows A_p as they were when the panel was factored
  // (later updates leave finished rows alone); so x_p = M^T (y_p - M s) = t_p - W_p s with
  // s = A_p,rest x_rest, t_p = M^T y_p and W_p = M^T M. W_p and t_p do not depend on the
  // solution, so they are formed for all panels at once, one panel per lane, leaving only
  // s and one 4-term product per panel on the serial path.
  {
    constexpr int kUsed = NPAN < 64 ? NPAN : 64;
    static_assert(NPAN <= 64, "one lane per panel");
    const int pl = lane < kUsed ? lane : kUsed - 1;
    if (4 * pl < D) {
      const float4 q0 = *reinterpret_cast<const float4 *>(&ud[pl][0]);
      const float4 q1 = *reinterpret_cast<const float4 *>(&ud[pl][4]);
      const float4 q2 = *reinterpret_cast<const float4 *>(&ud[pl][8]);
      const float4 q3 = *reinterpret_cast<const float4 *>(&ud[pl][12]);
      const float4 yy = *reinterpret_cast<const float4 *>(&ud[pl][16]);
      // M = [q0.x; q1.x q1.y; q2.x q2.y q2.z; q3.x q3.y q3.z q3.w] (lower triangular)
      const float w00 = q0.x * q0.x + q1.x * q1.x + q2.x * q2.x + q3.x * q3.x;
      const float w01 = q1.x * q1.y + q2.x * q2.y + q3.x * q3.y;
      const float w02 = q2.x * q2.z + q3.x * q3.z;
      const float w03 = q3.x * q3.w;
      const float w11 = q1.y * q1.y + q2.y * q2.y + q3.y * q3.y;
      const float w12 = q2.y * q2.z + q3.y * q3.z;
      const float w13 = q3.y * q3.w;
      const float w22 = q2.z * q2.z + q3.z * q3.z;
      const float w23 = q3.z * q3.w;
      const float w33 = q3.w * q3.w;
      const float t0 = q0.x * yy.x + q1.x * yy.y + q2.x * yy.z + q3.x * yy.w;
      const float t1 = q1.y * yy.y + q2.y * yy.z + q3.y * yy.w;
      const float t2 = q2.z * yy.z + q3.z * yy.w;
      const float t3 = q3.w * yy.w;
      if (lane < kUsed) {
        *reinterpret_cast<float4 *>(&ud[pl][0]) = make_float4(w00, w01, w02, w03);
        *reinterpret_cast<float4 *>(&ud[pl][4]) = make_float4(w01, w11, w12, w13);
        *reinterpret_cast<float4 *>(&ud[pl][8]) = make_float4(w02, w12, w22, w23);
        *reinterpret_cast<float4 *>(&ud[pl][12]) = make_float4(w03, w13, w23, w33);
        *reinterpret_cast<float4 *>(&ud[pl][16]) = make_float4(t0, t1, t2, t3);
      }
    }
    wave_sync();
  }
  float xv[T];
#pragma unroll
  for (int X = 0; X < T; ++X) xv[X] = 0.f;
#pragma unroll
  for (int I0 = T - 1; I0 >= 0; --I0) {
    // this tile row's partial products with the solved tiles X > I0 (row group g
    // holds panel g's rows; the 16-lane sums follow per panel), the newest tile last so
    // that one product per row waits for it
    float P0 = 0.f, P1 = 0.f, P2 = 0.f, P3 = 0.f;
#pragma unroll
    for (int X = T - 1; X > I0; --X) {
      const floatx4 aa = acc[tidx<T>(I0, X)];
      P0 = fmaf(aa[0], xv[X], P0);
      P1 = fmaf(aa[1], xv[X], P1);
      P2 = fmaf(aa[2], xv[X], P2);
      P3 = fmaf(aa[3], xv[X], P3);
    }
    // every lane's row of W_p and entry of t_p for the tile's four panels, read before the
    // serial steps (lane column 4 g + jj receives x[p0 + jj])
    float4 wrs[4];
    float tjs[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int pan = min(4 * I0 + g, NPAN - 1);
      const int jc = min(max(c - 4 * g, 0), 3);
      wrs[g] = *reinterpret_cast<const float4 *>(&ud[pan][4 * jc]);
      tjs[g] = ud[pan][16 + jc];
    }
#pragma unroll
    for (int g = 3; g >= 0; --g) {
      const int p0 = 16 * I0 + 4 * g;
      // panels of the tiles before the last are all inside D
      if (I0 == T - 1 && p0 >= D) continue;
      const int jj = c - 4 * g;
      const float4 wr = wrs[g];
      const float tj = tjs[g];
      // s_r = sum_{j > p0 + 3} A_p[r][j] x_j: the solved tiles plus the later panels
      // of this tile
      const float xj = c > 4 * g + 3 ? xv[I0] : 0.f;
      const floatx4 aa = acc[tidx<T>(I0, I0)];
      const float sr = sum16x4(fmaf(aa[0], xj, P0), fmaf(aa[1], xj, P1), fmaf(aa[2], xj, P2),
                               fmaf(aa[3], xj, P3));
      const float a0 = lane_value(sr, 16 * g + 0), a1 = lane_value(sr, 16 * g + 4);
      const float a2 = lane_value(sr, 16 * g + 8), a3 = lane_value(sr, 16 * g + 12);
      // computed in every lane and then selected: as a predicated update the compiler
      // moves the LDS reads of W_p and t_p into the serial step
      float x = tj - (fmaf(wr.x, a0, wr.y * a1) + fmaf(wr.z, a2, wr.w * a3));
      asm volatile("" : "+v"(x));
      xv[I0] = (jj >= 0 && jj < 4) ? x : xv[I0];
    }
  }

  // ---- write x (row group 0) unless flagged ----------------------------------------------------
  bool fin = true;
#pragma unroll
  for (int X = 0; X < T; ++X) fin &= (xv[X] == xv[X]) && fabsf(xv[X]) < INFINITY;
  bad |= __any(!fin) != 0;
  if (!bad) {
    if (kq == 0) {
#pragma unroll
      for (int X = 0; X < T; ++X)
        if (16 * X + c < D) xrow[16 * X + c] = xv[X];
    }
  } else if (lane == 0) {
    atomicAdd(flag_count, 1);
  }
  if (cyc_gram != nullptr && lane == 0) {
    const uint64_t t_end = __builtin_readcyclecounter();
    cyc_gram[task] = (double)(t_gram - t_start);
    cyc_solve[task] = (double)(t_end - t_gram);
  }
}

template <int DP>
static constexpr bool has_aug(int D) {
  return ((D + 3) & ~3) < DP;
}

template <int DP, bool AUG, bool WT, bool BAYES, bool TS = false, bool STRIP = false>
static void launch_rows_k(int64_t blocks, const RowTask *rows, int64_t n_rows,
                          const int32_t *idx, const uint8_t *val, const float *wts,
                          const float *Fp, int zrow, const float *ws, int D, float lam, float *X,
                          double *sse, int32_t *flag, double *cyc_gram, double *cyc_solve,
                          const RowPrior &pr, const Hadamard &hd, hipStream_t s) {
  hipLaunchKernelGGL((k_rows<DP, AUG, WT, BAYES, TS, STRIP>), dim3((unsigned)blocks),
                     dim3(64 * kRowWaves), 0, s, rows, n_rows, idx, val, wts, Fp, zrow, ws, D,
                     lam, X, sse, flag, cyc_gram, cyc_solve, pr, hd);
}

// The augmented variants, in strip form where the last tile uses four features.
template <int DP, bool WT, bool BAYES, bool TS, class... A>
static void launch_rows_aug(bool strip, A &&...args) {
  if constexpr (DP >= 48 && DP <= 112) {
    if (strip) return launch_rows_k<DP, true, WT, BAYES, TS, true>(args...);
  }
  launch_rows_k<DP, true, WT, BAYES, TS, false>(args...);
}

template <int DP>
static hipError_t launch_rows_t(const RowTask *rows, int64_t n_rows, const int32_t *idx,
                                const uint8_t *val, const float *wts, const float *Fp, int zrow,
                                const float *ws, int D, float lam, float *X, double *sse,
                                int32_t *flag, double *cyc_gram, double *cyc_solve,
                                const RowPrior &pr, const Hadamard &hd, hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  const int64_t blocks = (n_rows + kRowWaves - 1) / kRowWaves;
  const bool aug = has_aug<DP>(D), wt = wts != nullptr, strip = strip_width<DP>(D);
#define ROW_ARGS blocks, rows, n_rows, idx, val, wts, Fp, zrow, ws, D, lam, X, sse, flag, \
                 cyc_gram, cyc_solve, pr, hd, s
  if (hd.idx2) {
    // tensor ALS (and its Gibbs draws): no weights; the tile form throughout (with the
    // second gathered row the strip form needs more registers and is no faster)
    if (wt) return hipErrorInvalidValue;
    if (pr.init) {
      if (aug)
        launch_rows_k<DP, true, false, true, true>(ROW_ARGS);
      else
        launch_rows_k<DP, false, false, true, true>(ROW_ARGS);
    } else if (aug)
      launch_rows_k<DP, true, false, false, true>(ROW_ARGS);
    else
      launch_rows_k<DP, false, false, false, true>(ROW_ARGS);
  } else if (pr.init) {
    // the Gibbs half-sweep has no per-rating weights
    if (wt) return hipErrorInvalidValue;
    if (aug)
      launch_rows_aug<DP, false, true, false>(strip, ROW_ARGS);
    else
      launch_rows_k<DP, false, false, true>(ROW_ARGS);
  } else if (aug && wt)
    launch_rows_aug<DP, true, false, false>(strip, ROW_ARGS);
  else if (aug)
    launch_rows_aug<DP, false, false, false>(strip, ROW_ARGS);
  else if (wt)
    launch_rows_k<DP, false, true, false>(ROW_ARGS);
  else
    launch_rows_k<DP, false, false, false>(ROW_ARGS);
#undef ROW_ARGS
  return hipGetLastError();
}

template <int DP, bool AUG, bool WT, bool TS = false, bool STRIP = false>
static void launch_chunks_k(int64_t n, const WorkItem *items, const int32_t *idx,
                            const uint8_t *val, const float *wts, const float *Fp, int zrow,
                            const float *Xold, int D, float *ws, double *sse, const Hadamard &hd,
                            hipStream_t s) {
  hipLaunchKernelGGL((k_gram_chunks<DP, AUG, WT, TS, STRIP>), dim3((unsigned)n), dim3(64), 0, s,
                     items, idx, val, wts, Fp, zrow, Xold, D, ws, sse, hd);
}

template <int DP, bool WT, bool TS, class... A>
static void launch_chunks_aug(bool strip, A &&...args) {
  if constexpr (DP >= 48 && DP <= 112) {
    if (strip) return launch_chunks_k<DP, true, WT, TS, true>(args...);
  }
  launch_chunks_k<DP, true, WT, TS, false>(args...);
}

template <int DP>
static hipError_t launch_chunks_t(const WorkItem *items, int64_t n, const int32_t *idx,
                                  const uint8_t *val, const float *wts, const float *Fp,
                                  int zrow, const float *Xold, int D, float *ws, double *sse,
                                  const Hadamard &hd, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const bool aug = has_aug<DP>(D), wt = wts != nullptr, strip = strip_width<DP>(D);
#define CHUNK_ARGS n, items, idx, val, wts, Fp, zrow, Xold, D, ws, sse, hd, s
  if (hd.idx2) {
    if (wt) return hipErrorInvalidValue;
    if (aug)
      launch_chunks_k<DP, true, false, true>(CHUNK_ARGS);
    else
      launch_chunks_k<DP, false, false, true>(CHUNK_ARGS);
  } else if (aug && wt)
    launch_chunks_aug<DP, true, false>(strip, CHUNK_ARGS);
  else if (aug)
    launch_chunks_aug<DP, false, false>(strip, CHUNK_ARGS);
  else if (wt)
    launch_chunks_k<DP, false, true>(CHUNK_ARGS);
  else
    launch_chunks_k<DP, false, false>(CHUNK_ARGS);
#undef CHUNK_ARGS
  return hipGetLastError();
}

// Row kernels serve D > 20 (narrower widths take the one-lane solve).
#define ALS_DP_SWITCH(dp, CALL)                 \
  switch (dp) {                                 \
    case 32: { constexpr int DPV = 32; CALL; }  \
    case 48: { constexpr int DPV = 48; CALL; }  \
    case 64: { constexpr int DPV = 64; CALL; }  \
    case 80: { constexpr int DPV = 80; CALL; }  \
    case 96: { constexpr int DPV = 96; CALL; }  \
    case 112: { constexpr int DPV = 112; CALL; } \
    case 128: { constexpr int DPV = 128; CALL; } \
    default: return hipErrorInvalidValue;       \
  }

hipError_t launch_rows(int dp, const RowTask *rows, int64_t n_rows, const int32_t *idx,
                       const uint8_t *val, const float *wts, const float *Fp, int64_t n_fixed,
                       const float *ws, int D, float lam, float *X, double *sse, int32_t *flag,
                       double *cyc_gram, double *cyc_solve, const RowPrior &pr,
                       const Hadamard &hd, hipStream_t s) {
  if ((cyc_gram == nullptr) != (cyc_solve == nullptr)) return hipErrorInvalidValue;
  const int zrow = (int)n_fixed;
  ALS_DP_SWITCH(dp, return launch_rows_t<DPV>(rows, n_rows, idx, val, wts, Fp, zrow, ws, D, lam,
                                              X, sse, flag, cyc_gram, cyc_solve, pr, hd, s));
}

hipError_t launch_gram_chunks(int dp, const WorkItem *items, int64_t n, const int32_t *idx,
                              const uint8_t *val, const float *wts, const float *Fp,
                              int64_t n_fixed, const float *Xold, int D, float *ws, double *sse,
                              const Hadamard &hd, hipStream_t s) {
  const int zrow = (int)n_fixed;
  ALS_DP_SWITCH(dp, return launch_chunks_t<DPV>(items, n, idx, val, wts, Fp, zrow, Xold, D, ws,
                                                sse, hd, s));
}

}  // namespace als
