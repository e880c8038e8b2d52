// Regularise, factor and solve one row's normal equations in LDS (Sec. 2.2
// least-squares step; the per-update "matrix inversion" of Sec. 4.1 is done
// as a Cholesky factorisation A = L L^T and two triangular solves).
//
// One workgroup per row:
//  1. Sum the row's workspace slots in slot order (a split row has several),
//     scatter the upper-triangle Gram tiles into the lower triangle of A in
//     LDS, add lambda * n_s to the first D diagonal entries and 1 to the
//     padded ones (so padding factors as the identity and solves to zero).
//  2. Blocked right-looking Cholesky with 16-wide panels. For panel p:
//       a. one wavefront factors the 16x16 diagonal block (unblocked, LDS)
//          and forms its inverse Linv_p;
//       b. panel solve L_Ip = A_Ip Linv_p^T on MFMA (16x16x4, K = 16);
//       c. trailing update A_IJ -= L_Ip L_Jp^T on MFMA, tiles spread over the
//          wavefronts.
//  3. Blocked forward (L y = b) and backward (L^T x = y) solves by one
//     wavefront, using the stored Linv_p for the diagonal blocks.
//  4. If every pivot was positive and finite and x is finite, write x to the
//     row; otherwise leave the row unchanged and count it as flagged.
#include "internal.h"

namespace als {

typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Tile t of the row-major enumeration of upper-triangle tile pairs (I <= J).
template <int T>
__device__ __forceinline__ void tile_ij(int t, int &I, int &J) {
  I = 0;
  int rem = t;
  while (rem >= T - I) {
    rem -= T - I;
    ++I;
  }
  J = I + rem;
}

template <int DP, int NW>
__global__ __launch_bounds__(NW * 64) void k_chol(const RowTask *__restrict__ rows,
                                                  const float *__restrict__ ws, int D, float lam,
                                                  float *__restrict__ out,
                                                  int32_t *__restrict__ flag_count) {
  constexpr int T = DP / 16;
  constexpr int NT = T * (T + 1) / 2;
  constexpr int LDA = DP + 1;  // odd stride: column walks hit distinct banks
  constexpr int NTHR = NW * 64;
  constexpr int LI = 16 * 17;  // one stored 16x16 inverse, stride 17
  constexpr int64_t SLOT = (int64_t)slot_floats(DP);

  __shared__ float A[DP * LDA];
  __shared__ float Linv[T * LI];
  __shared__ float bv[DP];
  __shared__ float xv[DP];
  __shared__ float tv[16];
  __shared__ int bad;

  const RowTask rt = rows[blockIdx.x];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int kq = lane >> 4;
  const int c = lane & 15;

  if (tid == 0) bad = 0;

  // ---- 1. assemble A = G + lambda n I (lower triangle) and b ------------------------
  const float *__restrict__ base = ws + rt.slot0 * SLOT;
  for (int e = tid; e < NT * 256; e += NTHR) {
    float v = 0.f;
    for (int s = 0; s < rt.nslots; ++s) v += base[s * SLOT + e];
    const int t = e >> 8, ln = (e & 255) >> 2, r = e & 3;
    int I, J;
    tile_ij<T>(t, I, J);
    const int i = 16 * I + 4 * (ln >> 4) + r;  // Gram row
    const int j = 16 * J + (ln & 15);          // Gram column, j >= i for I < J
    A[j * LDA + i] = v;
  }
  for (int d = tid; d < DP; d += NTHR) {
    float v = 0.f;
    for (int s = 0; s < rt.nslots; ++s) v += base[s * SLOT + NT * 256 + d];
    bv[d] = v;
  }
  __syncthreads();
  const float lam_n = (float)((double)lam * (double)rt.deg);
  for (int d = tid; d < DP; d += NTHR) A[d * LDA + d] = d < D ? A[d * LDA + d] + lam_n : 1.0f;
  __syncthreads();

  // ---- 2. blocked Cholesky ------------------------------------------------------------
  for (int p = 0; p < T; ++p) {
    const int p0 = 16 * p;
    if (w == 0) {
      for (int kk = 0; kk < 16; ++kk) {
        const float piv = A[(p0 + kk) * LDA + p0 + kk];
        const bool okp = piv > 0.f && piv < INFINITY;
        if (!okp && lane == 0) bad = 1;
        const float dg = sqrtf(okp ? piv : 1.f);
        const float inv = 1.f / dg;
        if (lane < 16) {
          if (lane > kk) A[(p0 + lane) * LDA + p0 + kk] *= inv;
          else if (lane == kk) A[(p0 + kk) * LDA + p0 + kk] = dg;
        }
        wave_sync();
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int ii = 4 * kq + r;
          if (c > kk && ii >= c)
            A[(p0 + ii) * LDA + p0 + c] -=
                A[(p0 + ii) * LDA + p0 + kk] * A[(p0 + c) * LDA + p0 + kk];
        }
        wave_sync();
      }
      if (lane < 16) {
        float x[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          float s = (i == c) ? 1.f : 0.f;
#pragma unroll
          for (int m = 0; m < i; ++m) s -= A[(p0 + i) * LDA + p0 + m] * x[m];
          x[i] = (i >= c) ? s / A[(p0 + i) * LDA + p0 + i] : 0.f;
        }
#pragma unroll
        for (int i = 0; i < 16; ++i) Linv[p * LI + i * 17 + c] = x[i];
      }
    }
    __syncthreads();
    // panel: L_Ip = A_Ip Linv_p^T
    for (int I = p + 1 + w; I < T; I += NW) {
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4) {
        const float a = A[(16 * I + c) * LDA + p0 + 4 * s4 + kq];
        const float b = Linv[p * LI + c * 17 + 4 * s4 + kq];
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) A[(16 * I + 4 * kq + r) * LDA + p0 + c] = acc[r];
    }
    __syncthreads();
    // trailing update: A_IJ -= L_Ip L_Jp^T for p < J <= I
    const int m = T - 1 - p;
    const int npairs = m * (m + 1) / 2;
    for (int q = w; q < npairs; q += NW) {
      int J = p + 1, rem = q;
      while (rem >= T - J) {
        rem -= T - J;
        ++J;
      }
      const int I = J + rem;
      floatx4 acc;
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r] = A[(16 * I + 4 * kq + r) * LDA + 16 * J + c];
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4) {
        const float a = -A[(16 * I + c) * LDA + p0 + 4 * s4 + kq];
        const float b = A[(16 * J + c) * LDA + p0 + 4 * s4 + kq];
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) A[(16 * I + 4 * kq + r) * LDA + 16 * J + c] = acc[r];
    }
    __syncthreads();
  }

  // ---- 3. triangular solves (one wavefront) -----------------------------------------------
  if (w == 0) {
    for (int p = 0; p < T; ++p) {  // forward: y = L^{-1} b
      const int p0 = 16 * p;
      float s = 0.f;
      for (int mm = kq; mm < p0; mm += 4) s += A[(p0 + c) * LDA + mm] * xv[mm];
      s += __shfl_xor(s, 16);
      s += __shfl_xor(s, 32);
      if (lane < 16) tv[c] = bv[p0 + c] - s;
      wave_sync();
      float y = 0.f;
#pragma unroll
      for (int jj = kq; jj < 16; jj += 4) y += Linv[p * LI + c * 17 + jj] * tv[jj];
      y += __shfl_xor(y, 16);
      y += __shfl_xor(y, 32);
      if (lane < 16) xv[p0 + c] = y;
      wave_sync();
    }
    for (int p = T - 1; p >= 0; --p) {  // backward: x = L^{-T} y
      const int p0 = 16 * p;
      float s = 0.f;
      for (int mm = p0 + 16 + kq; mm < DP; mm += 4) s += A[mm * LDA + p0 + c] * xv[mm];
      s += __shfl_xor(s, 16);
      s += __shfl_xor(s, 32);
      if (lane < 16) tv[c] = xv[p0 + c] - s;
      wave_sync();
      float x = 0.f;
#pragma unroll
      for (int jj = kq; jj < 16; jj += 4) x += Linv[p * LI + jj * 17 + c] * tv[jj];
      x += __shfl_xor(x, 16);
      x += __shfl_xor(x, 32);
      if (lane < 16) xv[p0 + c] = x;
      wave_sync();
    }
  }
  __syncthreads();

  // ---- 4. write or flag ---------------------------------------------------------------------
  for (int d = tid; d < D; d += NTHR) {
    const float x = xv[d];
    if (!(x == x) || x == INFINITY || x == -INFINITY) bad = 1;
  }
  __syncthreads();
  if (!bad) {
    for (int d = tid; d < D; d += NTHR) out[(int64_t)rt.row * D + d] = xv[d];
  } else if (tid == 0) {
    atomicAdd(flag_count, 1);
  }
}

template <int DP, int NW>
static hipError_t launch_chol_t(const RowTask *rows, int64_t n_rows, const float *ws, int D,
                                float lam, float *out, int32_t *flag_count, hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  hipLaunchKernelGGL((k_chol<DP, NW>), dim3((unsigned)n_rows), dim3(NW * 64), 0, s, rows, ws, D,
                     lam, out, flag_count);
  return hipGetLastError();
}

hipError_t launch_chol(int dp, const RowTask *rows, int64_t n_rows, const float *ws, int D,
                       float lam, float *out, int32_t *flag_count, hipStream_t s) {
  switch (dp) {
    case 16: return launch_chol_t<16, 1>(rows, n_rows, ws, D, lam, out, flag_count, s);
    case 32: return launch_chol_t<32, 1>(rows, n_rows, ws, D, lam, out, flag_count, s);
    case 48: return launch_chol_t<48, 4>(rows, n_rows, ws, D, lam, out, flag_count, s);
    case 64: return launch_chol_t<64, 4>(rows, n_rows, ws, D, lam, out, flag_count, s);
    case 80: return launch_chol_t<80, 4>(rows, n_rows, ws, D, lam, out, flag_count, s);
    case 96: return launch_chol_t<96, 4>(rows, n_rows, ws, D, lam, out, flag_count, s);
    case 112: return launch_chol_t<112, 4>(rows, n_rows, ws, D, lam, out, flag_count, s);
    case 128: return launch_chol_t<128, 4>(rows, n_rows, ws, D, lam, out, flag_count, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace als
