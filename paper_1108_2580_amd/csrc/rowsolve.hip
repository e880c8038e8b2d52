// The fused row kernel of the ALS half-sweep (Sec. 2.2): for each row s of the
// solved side, one wavefront
//   1. accumulates the normal equations G = sum_k f_k f_k^T (upper-triangle
//      16x16 tiles, fp32 MFMA 16x16x4, held in accumulator registers) and
//      b = sum_k r_k f_k over the row's ratings, and on the same gathered rows
//      the squared residuals (r_k - x_s . f_k)^2 of the state entering the
//      half-sweep (x_s = the row's previous value) for the training RMSE
//      (Sec. 4.1);
//   2. factors A = U^T U (lambda n_s I is the accumulators' initial value) in
//      panels of four rows: the 4x4 diagonal block is factored in every lane,
//      the panel rows of U are formed by a 4x4 triangular solve per column, and
//      the trailing tiles are updated on MFMA (K = 4). The accumulators are only
//      written by MFMA and read by VALU, so they stay in accumulator registers;
//   3. forward substitution of b rides along the panels; back substitution
//      follows, forming U's panel rows from the untouched A_p rows and the
//      stored 4x4 blocks; x_s is written unless a pivot was not positive and
//      finite.
// Rows with more ratings than the hub threshold have their normal equations
// built by several wavefronts (k_gram_chunks, partials in a workspace) and are
// only summed and solved here.
//
// Register layout: lane (kq, c) = (lane / 16, lane % 16). Gram operand block X
// of rating k is feature 16 X + c of f_k in lane (k, c). Accumulator tile
// (I, J), I <= J, holds A[16 I + 4 kq + r][16 J + c] in element r. The fixed
// side is read from a staged copy with row stride DP (zero padded), so every
// gathered row starts on a 64-byte boundary.
#include "gram.h"

namespace als {

// Copy the fixed factors [n x D] into a zero-padded [(n + 1) x DP] buffer whose
// last row is all zero (the stand-in of padded features and absent ratings).
__global__ void k_stage_fixed(const float *__restrict__ F, int64_t n, int D, int DP,
                              float *__restrict__ Fp) {
  const int64_t total = (n + 1) * DP;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < total; i += stride) {
    const int64_t row = i / DP;
    const int d = (int)(i - row * DP);
    Fp[i] = (row < n && d < D) ? F[row * D + d] : 0.f;
  }
}

hipError_t launch_stage_fixed(const float *F, int64_t n, int D, int DP, float *Fp, hipStream_t s) {
  if (n < 0) return hipErrorInvalidValue;
  int64_t blocks = ((n + 1) * DP + 255) / 256;
  if (blocks > 262144) blocks = 262144;
  hipLaunchKernelGGL(k_stage_fixed, dim3((unsigned)blocks), dim3(256), 0, s, F, n, D, DP, Fp);
  return hipGetLastError();
}

// Partial normal equations of the chunks of split rows, with the chunks'
// entering-state squared residuals.
template <int DP>
__global__ __launch_bounds__(64) void k_gram_chunks(const WorkItem *__restrict__ items,
                                                    const int32_t *__restrict__ idx,
                                                    const uint8_t *__restrict__ val,
                                                    const float *__restrict__ Fp, int zrow,
                                                    const float *__restrict__ Xold, int D,
                                                    float *__restrict__ ws,
                                                    double *__restrict__ sse_out) {
  using C = RowCfg<DP>;
  constexpr int T = C::T, NT = C::NT;
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
  gram_accumulate<DP>(acc, rhs, xo, sse, idx + it.start, val + it.start, it.len, Fp, zrow, D);
#pragma unroll
  for (int X = 0; X < T; ++X) {
    rhs[X] += __shfl_xor(rhs[X], 16);
    rhs[X] += __shfl_xor(rhs[X], 32);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sse += __shfl_xor(sse, o);
  float *__restrict__ out = ws + it.slot * (int64_t)slot_floats(DP);
#pragma unroll
  for (int t = 0; t < NT; ++t) *reinterpret_cast<floatx4 *>(out + t * 256 + lane * 4) = acc[t];
  if (kq == 0) {
#pragma unroll
    for (int X = 0; X < T; ++X) out[NT * 256 + 16 * X + c] = rhs[X];
  }
  if (lane == 0) sse_out[blockIdx.x] = sse;
}

constexpr int kRowWaves = 4;  // independent rows per workgroup (one per wavefront)

// Two wavefronts per SIMD (the second launch bound) outweigh the few registers the
// wide widths then spill: the accumulator tiles move to arch VGPRs and the gather
// latency of one row hides behind the other row's MFMAs.

template <int DP>
__global__ __launch_bounds__(64 * kRowWaves, 2) void k_rows(
    const RowTask *__restrict__ rows, int64_t n_rows, const int32_t *__restrict__ idx,
    const uint8_t *__restrict__ val, const float *__restrict__ Fp, int zrow,
    const float *__restrict__ ws, int D, float lam, float *__restrict__ X_io,
    double *__restrict__ sse_out,
    int32_t *__restrict__ flag_count) {
  using C = RowCfg<DP>;
  constexpr int T = C::T, NT = C::NT;
  constexpr int NPAN = DP / 4;
  __shared__ floatx4 s_panel[kRowWaves][T][16];  // one panel's rows, per tile column and lane column
  __shared__ float s_ud[kRowWaves][NPAN][12];    // per panel: 4x4 U block (10) + spare

  const int wv = threadIdx.x >> 6;
  const int64_t task = (int64_t)blockIdx.x * kRowWaves + wv;
  if (task >= n_rows) return;
  const RowTask rt = rows[task];
  const int lane = threadIdx.x & 63, kq = lane >> 4, c = lane & 15;
  floatx4(&panel)[T][16] = s_panel[wv];
  float(&ud)[NPAN][12] = s_ud[wv];

  // A starts as lambda n_s I on the first D diagonal entries and I on the padding;
  // the Gram (or the sum of a split row's chunk partials) is accumulated on top
  const float lam_n = (float)((double)lam * (double)rt.deg);
  floatx4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int I = 0; I < T; ++I) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int d = 16 * I + 4 * kq + r;
      acc[tidx<T>(I, I)][r] = c == 4 * kq + r ? (d < D ? lam_n : 1.f) : 0.f;
    }
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
    gram_accumulate<DP>(acc, rhs, xo, sse, idx + rt.start, val + rt.start, rt.deg, Fp, zrow, D);
#pragma unroll
    for (int X = 0; X < T; ++X) {
      rhs[X] += __shfl_xor(rhs[X], 16);
      rhs[X] += __shfl_xor(rhs[X], 32);
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
#pragma unroll
      for (int X = 0; X < T; ++X) rhs[X] += sl[NT * 256 + 16 * X + c];
    }
  }

  // ---- factorisation A = U^T U with forward substitution U^T y = b ------------------------
  bool bad = false;
#pragma unroll
  for (int I0 = 0; I0 < T; ++I0) {
    // panels of one tile row run as a loop (unrolling them all would blow up the
    // register allocation around the accumulator tiles)
#pragma clang loop unroll(disable)
    for (int g = 0; g < 4; ++g) {
      const int p0 = 16 * I0 + 4 * g;
      if (p0 >= D) break;
      // (1) publish the panel rows p0..p0+3 (held by row group g)
      if (kq == g) {
#pragma unroll
        for (int X = I0; X < T; ++X) panel[X][c] = acc[tidx<T>(I0, X)];
      }
      wave_sync();
      // (2) 4x4 diagonal block, factored redundantly in every lane
      const floatx4 d0 = panel[I0][4 * g + 0], d1 = panel[I0][4 * g + 1];
      const floatx4 d2 = panel[I0][4 * g + 2], d3 = panel[I0][4 * g + 3];
      // d{r'}[r] = A[p0 + r][p0 + r']
      const float a00 = d0[0], a01 = d1[0], a02 = d2[0], a03 = d3[0];
      const float a11 = d1[1], a12 = d2[1], a13 = d3[1];
      const float a22 = d2[2], a23 = d3[2], a33 = d3[3];
      float p;
      p = a00;
      bad |= !(p > 0.f && p < INFINITY);
      const float i00 = inv_sqrt_pivot(p);
      const float u01 = a01 * i00, u02 = a02 * i00, u03 = a03 * i00;
      p = a11 - u01 * u01;
      bad |= !(p > 0.f && p < INFINITY);
      const float i11 = inv_sqrt_pivot(p);
      const float u12 = (a12 - u01 * u02) * i11, u13 = (a13 - u01 * u03) * i11;
      p = a22 - u02 * u02 - u12 * u12;
      bad |= !(p > 0.f && p < INFINITY);
      const float i22 = inv_sqrt_pivot(p);
      const float u23 = (a23 - u02 * u03 - u12 * u13) * i22;
      p = a33 - u03 * u03 - u13 * u13 - u23 * u23;
      bad |= !(p > 0.f && p < INFINITY);
      const float i33 = inv_sqrt_pivot(p);
      const int pan = p0 >> 2;
      if (lane == 0) {
        ud[pan][0] = i00; ud[pan][1] = u01; ud[pan][2] = u02; ud[pan][3] = u03;
        ud[pan][4] = i11; ud[pan][5] = u12; ud[pan][6] = u13;
        ud[pan][7] = i22; ud[pan][8] = u23; ud[pan][9] = i33;
      }
      // right-hand side of the panel rows, from lanes c = 4g + r
      const float b0 = lane_value(rhs[I0], 4 * g + 0), b1 = lane_value(rhs[I0], 4 * g + 1);
      const float b2 = lane_value(rhs[I0], 4 * g + 2), b3 = lane_value(rhs[I0], 4 * g + 3);
      const float y0 = b0 * i00;
      const float y1 = (b1 - u01 * y0) * i11;
      const float y2 = (b2 - u02 * y0 - u12 * y1) * i22;
      const float y3 = (b3 - u03 * y0 - u13 * y1 - u23 * y2) * i33;
      // (3) panel rows U[p0 + q][j] = (U^{-T} A[p0.., j])_q and trailing operands
      float u[T];
#pragma unroll
      for (int X = 0; X < T; ++X) {
        u[X] = 0.f;
        if (X >= I0) {
          const floatx4 col = panel[X][c];
          const float Y0 = col[0] * i00;
          const float Y1 = (col[1] - u01 * Y0) * i11;
          const float Y2 = (col[2] - u02 * Y0 - u12 * Y1) * i22;
          const float Y3 = (col[3] - u03 * Y0 - u13 * Y1 - u23 * Y2) * i33;
          const int j = 16 * X + c;
          if (j > p0 + 3) {
            u[X] = kq == 0 ? Y0 : (kq == 1 ? Y1 : (kq == 2 ? Y2 : Y3));
            rhs[X] -= Y0 * y0 + Y1 * y1 + Y2 * y2 + Y3 * y3;
          } else if (j >= p0) {
            rhs[X] = j == p0 ? y0 : (j == p0 + 1 ? y1 : (j == p0 + 2 ? y2 : y3));
          }
        }
      }
      // (4) trailing update on MFMA: A_IJ -= U_p(:, I)^T U_p(:, J). The tile row that the
      // next panel publishes is issued first, so that the next panel's factorisation runs
      // while the matrix unit works through the rest. After the last panel of a tile row
      // (g == 3) that row has no unfactored rows left and its update is skipped.
      if (g < 3) {
#pragma unroll
        for (int J = I0; J < T; ++J)
          acc[tidx<T>(I0, J)] =
              __builtin_amdgcn_mfma_f32_16x16x4f32(-u[I0], u[J], acc[tidx<T>(I0, J)], 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int I = I0 + 1; I < T; ++I) {
#pragma unroll
        for (int J = I; J < T; ++J)
          acc[tidx<T>(I, J)] =
              __builtin_amdgcn_mfma_f32_16x16x4f32(-u[I], u[J], acc[tidx<T>(I, J)], 0, 0, 0);
      }
      wave_sync();
    }
  }

  // ---- back substitution U x = y (rhs holds y) ----------------------------------------------
  float xv[T];
#pragma unroll
  for (int X = 0; X < T; ++X) xv[X] = 0.f;
#pragma unroll
  for (int I0 = T - 1; I0 >= 0; --I0) {
#pragma clang loop unroll(disable)
    for (int g = 3; g >= 0; --g) {
      const int p0 = 16 * I0 + 4 * g;
      if (p0 >= D) continue;
      // s_r = sum_{j > p0 + 3} A_p[r][j] x_j, partials in row group g
      float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
#pragma unroll
      for (int X = I0; X < T; ++X) {
        const int j = 16 * X + c;
        const float xj = j > p0 + 3 ? xv[X] : 0.f;
        const floatx4 uu = acc[tidx<T>(I0, X)];
        s0 = fmaf(uu[0], xj, s0);
        s1 = fmaf(uu[1], xj, s1);
        s2 = fmaf(uu[2], xj, s2);
        s3 = fmaf(uu[3], xj, s3);
      }
      s0 = sum16(s0);
      s1 = sum16(s1);
      s2 = sum16(s2);
      s3 = sum16(s3);
      const float a0 = lane_value(s0, 16 * g), a1 = lane_value(s1, 16 * g);
      const float a2 = lane_value(s2, 16 * g), a3 = lane_value(s3, 16 * g);
      const float y0 = lane_value(rhs[I0], 4 * g + 0), y1 = lane_value(rhs[I0], 4 * g + 1);
      const float y2 = lane_value(rhs[I0], 4 * g + 2), y3 = lane_value(rhs[I0], 4 * g + 3);
      const int pan = p0 >> 2;
      const float i00 = ud[pan][0], u01 = ud[pan][1], u02 = ud[pan][2], u03 = ud[pan][3];
      const float i11 = ud[pan][4], u12 = ud[pan][5], u13 = ud[pan][6];
      const float i22 = ud[pan][7], u23 = ud[pan][8], i33 = ud[pan][9];
      // the accumulators still hold the panel rows A_p as they were when the panel
      // was factored, and U's panel rows are U_gg^{-T} A_p, so
      // sum_j U[p0 + r][j] x_j = (U_gg^{-T} (A_p x))_r
      const float t0 = a0 * i00;
      const float t1 = (a1 - u01 * t0) * i11;
      const float t2 = (a2 - u02 * t0 - u12 * t1) * i22;
      const float t3 = (a3 - u03 * t0 - u13 * t1 - u23 * t2) * i33;
      const float x3 = (y3 - t3) * i33;
      const float x2 = (y2 - t2 - u23 * x3) * i22;
      const float x1 = (y1 - t1 - u12 * x2 - u13 * x3) * i11;
      const float x0 = (y0 - t0 - u01 * x1 - u02 * x2 - u03 * x3) * i00;
      const int jj = c - 4 * g;
      if (jj >= 0 && jj < 4) xv[I0] = jj == 0 ? x0 : (jj == 1 ? x1 : (jj == 2 ? x2 : x3));
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
}

template <int DP>
static hipError_t launch_rows_t(const RowTask *rows, int64_t n_rows, const int32_t *idx,
                                const uint8_t *val, const float *Fp, int zrow, const float *ws,
                                int D, float lam, float *X, double *sse, int32_t *flag,
                                hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  const int64_t blocks = (n_rows + kRowWaves - 1) / kRowWaves;
  hipLaunchKernelGGL(k_rows<DP>, dim3((unsigned)blocks), dim3(64 * kRowWaves), 0, s, rows, n_rows,
                     idx, val, Fp, zrow, ws, D, lam, X, sse, flag);
  return hipGetLastError();
}

template <int DP>
static hipError_t launch_chunks_t(const WorkItem *items, int64_t n, const int32_t *idx,
                                  const uint8_t *val, const float *Fp, int zrow,
                                  const float *Xold, int D, float *ws, double *sse,
                                  hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_gram_chunks<DP>, dim3((unsigned)n), dim3(64), 0, s, items, idx, val, Fp,
                     zrow, Xold, D, ws, sse);
  return hipGetLastError();
}

#define ALS_DP_SWITCH(dp, CALL)                 \
  switch (dp) {                                 \
    case 16: { constexpr int DPV = 16; CALL; }  \
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
                       const uint8_t *val, const float *Fp, int64_t n_fixed, const float *ws,
                       int D, float lam, float *X, double *sse, int32_t *flag, hipStream_t s) {
  const int zrow = (int)n_fixed;
  ALS_DP_SWITCH(dp, return launch_rows_t<DPV>(rows, n_rows, idx, val, Fp, zrow, ws, D, lam, X,
                                              sse, flag, s));
}

hipError_t launch_gram_chunks(int dp, const WorkItem *items, int64_t n, const int32_t *idx,
                              const uint8_t *val, const float *Fp, int64_t n_fixed,
                              const float *Xold, int D, float *ws, double *sse, hipStream_t s) {
  const int zrow = (int)n_fixed;
  ALS_DP_SWITCH(dp, return launch_chunks_t<DPV>(items, n, idx, val, Fp, zrow, Xold, D, ws, sse,
                                                s));
}

}  // namespace als
