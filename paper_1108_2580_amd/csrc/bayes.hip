// Bayesian factorisation (BPTF, named in Sec. 2.2: least squares plus sampling from the
// hyperpriors of U and V), in the form of the published BPMF / BPTF Gibbs sampler.
// Ratings are Gaussian with precision alpha around u . v; each row of a side has the
// prior N(mu, Lambda^{-1}); (mu, Lambda) has a Normal-Wishart hyperprior. The row draws
// reuse the half-sweep kernels (their BAYES variants): this file holds the rest.
//
//   k_prior_prepare   one workgroup, fp64: the prior image the row kernels start from
//                     (Lambda / alpha with the identity on the padding, and
//                     Lambda mu / alpha), laid out as a workspace slot (D > 20) or a
//                     packed record (D <= 20); and K = L^{-T} (Lambda = L L^T) for the
//                     rows without ratings, which are drawn from the prior.
//   k_prior_rows      one lane per row without ratings: x = mu + K z.
//   k_hyper_moments   per-block fp64 sums of x and of the upper triangle of x x^T over
//                     the side's rows (rows staged through LDS); products of two fp32
//                     values are exact in fp64, so only the summation order rounds.
//   k_hyper_sample    one workgroup, fp64: sums the blocks in order, forms the
//                     Normal-Wishart posterior (beta* = beta0 + n, nu* = nu0 + n,
//                     mu0* = (beta0 mu0 + n xbar) / beta*, W*^{-1} = W0^{-1} + S +
//                     beta0 n / beta* (mu0 - xbar)(mu0 - xbar)^T with S the scatter
//                     about the mean), then Bartlett's draw: W* = F F^T, B lower
//                     triangular with B_ii = sqrt(chi2_i) and normal B_ij, Lambda =
//                     (F B)(F B)^T, and mu = mu0* + R^{-T} zmu with beta* Lambda = R R^T.
// The variates (chi-square, normals) are inputs. Matrices live in the fp64 scratch as
// full row-major D x D arrays; the factorisations are right-looking Cholesky steps with
// a barrier between steps.
#include "internal.h"

namespace als {

namespace {

constexpr int kBayesBlock = 256;
constexpr int kMomentRows = 32;  // rows per LDS stage of the moment kernel
constexpr int kMaxEntriesPerThread = (128 + 128 * 129 / 2 + kBayesBlock - 1) / kBayesBlock;
constexpr int kHyperBlocks = 1024;

// In-place lower Cholesky factor of the D x D matrix A (the lower triangle is read, the
// strict upper triangle is zeroed). *bad is set when a pivot is not positive and finite.
__device__ void blk_cholesky(double *A, int D, int *bad) {
  for (int k = 0; k < D; ++k) {
    __syncthreads();
    const double p = A[k * D + k];
    const bool ok = p > 0.0 && isfinite(p);
    const double l = sqrt(ok ? p : 1.0);
    if (!ok && threadIdx.x == 0) *bad = 1;
    __syncthreads();
    if (threadIdx.x == 0) A[k * D + k] = l;
    for (int i = k + 1 + threadIdx.x; i < D; i += blockDim.x) A[i * D + k] /= l;
    __syncthreads();
    const int m = D - k - 1;
    for (int q = threadIdx.x; q < m * m; q += blockDim.x) {
      const int i = k + 1 + q / m, j = k + 1 + q % m;
      if (j <= i) A[i * D + j] -= A[i * D + k] * A[j * D + k];
    }
  }
  __syncthreads();
  for (int q = threadIdx.x; q < D * D; q += blockDim.x)
    if (q % D > q / D) A[q] = 0.0;
  __syncthreads();
}

// Li = L^{-1} (lower triangular), one column per thread.
__device__ void blk_lower_inverse(const double *L, double *Li, int D) {
  for (int e = threadIdx.x; e < D; e += blockDim.x) {
    for (int i = 0; i < D; ++i) {
      if (i < e) {
        Li[i * D + e] = 0.0;
        continue;
      }
      double s = i == e ? 1.0 : 0.0;
      for (int m = e; m < i; ++m) s -= L[i * D + m] * Li[m * D + e];
      Li[i * D + e] = s / L[i * D + i];
    }
  }
  __syncthreads();
}

// C = A B^T for full D x D matrices (C distinct from A and B).
__device__ void blk_mul_abt(const double *A, const double *B, double *C, int D) {
  for (int q = threadIdx.x; q < D * D; q += blockDim.x) {
    const int i = q / D, j = q % D;
    double t = 0.0;
    for (int m = 0; m < D; ++m) t += A[i * D + m] * B[j * D + m];
    C[q] = t;
  }
  __syncthreads();
}

__global__ __launch_bounds__(kBayesBlock) void k_prior_prepare(
    const double *__restrict__ Lam, const double *__restrict__ mu, int D, int DP, int LD,
    int aug_col, double alpha, float *__restrict__ init, float *__restrict__ K,
    float *__restrict__ mu32, double *__restrict__ scratch, int32_t *__restrict__ ok) {
  __shared__ int bad;
  if (threadIdx.x == 0) bad = 0;
  double *c = scratch;            // Lambda mu / alpha
  double *L = scratch + 2 * D;    // Cholesky factor of Lambda
  double *Li = L + D * D;         // its inverse
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    double t = 0.0;
    for (int e = 0; e < D; ++e) t += Lam[d * D + e] * mu[e];
    c[d] = t / alpha;
    mu32[d] = (float)mu[d];
  }
  for (int q = threadIdx.x; q < D * D; q += blockDim.x) L[q] = Lam[q];
  __syncthreads();
  // entry (r, col) of the scaled prior matrix, the identity on the padding, and with the
  // augmented column (D > 20 only) holding Lambda mu / alpha
  auto entry = [&](int r, int col) -> float {
    if (r < D && col < D) return (float)(Lam[r * D + col] / alpha);
    if (col == aug_col && r < D) return (float)c[r];
    return r == col ? 1.f : 0.f;
  };
  if (LD > 0) {
    const int ntri = LD * (LD + 1) / 2, total = ne_floats(LD);
    for (int q = threadIdx.x; q < total; q += blockDim.x) {
      float v = 0.f;
      if (q < ntri) {
        int a = 0, rem = q;
        while (rem >= LD - a) {
          rem -= LD - a;
          ++a;
        }
        v = entry(a, a + rem);
      } else if (q < ntri + LD) {
        const int d = q - ntri;
        v = d < D ? (float)c[d] : 0.f;
      }
      init[q] = v;
    }
  } else {
    const int T = DP / 16, NT = T * (T + 1) / 2;
    const int total = NT * 256 + DP;
    for (int q = threadIdx.x; q < total; q += blockDim.x) {
      float v = 0.f;
      if (q < NT * 256) {
        int t = q >> 8, I = 0;
        while (t >= T - I) {
          t -= T - I;
          ++I;
        }
        const int J = I + t, lane = (q & 255) >> 2, r = q & 3;
        v = entry(16 * I + 4 * (lane >> 4) + r, 16 * J + (lane & 15));
      } else {
        const int d = q - NT * 256;
        v = (aug_col < 0 && d < D) ? (float)c[d] : 0.f;
      }
      init[q] = v;
    }
  }
  // K = L^{-T} for the rows without ratings
  blk_cholesky(L, D, &bad);
  blk_lower_inverse(L, Li, D);
  for (int q = threadIdx.x; q < D * D; q += blockDim.x) K[q] = (float)Li[(q % D) * D + q / D];
  __syncthreads();
  if (threadIdx.x == 0) *ok = bad ? 0 : 1;
}

__global__ __launch_bounds__(64) void k_prior_rows(const int32_t *__restrict__ rows, int64_t n,
                                                  int D, const float *__restrict__ K,
                                                  const float *__restrict__ mu32,
                                                  const int32_t *__restrict__ ok,
                                                  const float *__restrict__ z,
                                                  float *__restrict__ X,
                                                  int32_t *__restrict__ flag_count) {
  const int64_t i = (int64_t)blockIdx.x * 64 + threadIdx.x;
  if (i >= n) return;
  const int64_t row = rows[i];
  if (*ok == 0) {
    atomicAdd(flag_count, 1);
    return;
  }
  const float *__restrict__ zr = z + row * D;
  float *__restrict__ xr = X + row * D;
  for (int a = 0; a < D; ++a) {
    float t = mu32[a];
    for (int e = a; e < D; ++e) t = fmaf(K[a * D + e], zr[e], t);
    xr[a] = t;
  }
}

__global__ __launch_bounds__(kBayesBlock) void k_hyper_moments(const float *__restrict__ X,
                                                               int64_t n, int D,
                                                               double *__restrict__ partials) {
  __shared__ float xs[kMomentRows][128];
  const int ne = D + D * (D + 1) / 2;
  // this thread's entries: packed (a, e) pairs, e = a + (upper triangle) or e = -1 (sum of x_a)
  int16_t ea[kMaxEntriesPerThread], ee[kMaxEntriesPerThread];
  double acc[kMaxEntriesPerThread];
  int cnt = 0;
#pragma unroll
  for (int k = 0; k < kMaxEntriesPerThread; ++k) {
    const int q = threadIdx.x + k * kBayesBlock;
    ea[k] = 0;
    ee[k] = -1;
    acc[k] = 0.0;
    if (q < ne) {
      cnt = k + 1;
      if (q < D) {
        ea[k] = (int16_t)q;
      } else {
        int rem = q - D, a = 0;
        while (rem >= D - a) {
          rem -= D - a;
          ++a;
        }
        ea[k] = (int16_t)a;
        ee[k] = (int16_t)(a + rem);
      }
    }
  }
  const int64_t per = (n + gridDim.x - 1) / gridDim.x;
  const int64_t r0 = (int64_t)blockIdx.x * per, r1 = min(n, r0 + per);
  for (int64_t base = r0; base < r1; base += kMomentRows) {
    const int rows = (int)min<int64_t>(kMomentRows, r1 - base);
    __syncthreads();
    for (int q = threadIdx.x; q < rows * D; q += kBayesBlock)
      xs[q / D][q % D] = X[(base + q / D) * D + q % D];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kMaxEntriesPerThread; ++k) {
      if (k < cnt) {
        const int a = ea[k], e = ee[k];
        double t = acc[k];
        if (e < 0) {
          for (int r = 0; r < rows; ++r) t += (double)xs[r][a];
        } else {
          for (int r = 0; r < rows; ++r) t = fma((double)xs[r][a], (double)xs[r][e], t);
        }
        acc[k] = t;
      }
    }
  }
#pragma unroll
  for (int k = 0; k < kMaxEntriesPerThread; ++k) {
    const int q = threadIdx.x + k * kBayesBlock;
    if (q < ne) partials[(int64_t)blockIdx.x * ne + q] = acc[k];
  }
}

__global__ __launch_bounds__(kBayesBlock) void k_hyper_sample(
    const double *__restrict__ partials, int nblk, int64_t n, int D,
    const double *__restrict__ mu0, double beta0, const double *__restrict__ W0inv, double nu0,
    const double *__restrict__ chi2, const double *__restrict__ offd,
    const double *__restrict__ zmu, double *__restrict__ scratch, double *__restrict__ mu_out,
    double *__restrict__ Lam_out, int32_t *__restrict__ status) {
  __shared__ int bad;
  if (threadIdx.x == 0) bad = 0;
  const int ne = D + D * (D + 1) / 2, DD = D * D;
  double *A = scratch;        // W*^{-1}, then its factor R
  double *B = A + DD;         // R^{-1}
  double *C = B + DD;         // W*, then its factor F
  double *E = C + DD;         // F B
  double *G = E + DD;         // beta* Lambda, then its factor
  double *H = G + DD;         // moments: sums of x_a, then of x_a x_e (upper triangle)
  double *xbar = H + ne;      // mean, then mu0*
  double *dv = xbar + D;      // mu0 - xbar
  double *tmp = dv + D;
  for (int q = threadIdx.x; q < ne; q += blockDim.x) {
    double t = 0.0;
    for (int b = 0; b < nblk; ++b) t += partials[(int64_t)b * ne + q];
    H[q] = t;
  }
  __syncthreads();
  const double nn = (double)n;
  const double beta_s = beta0 + nn, nu_s = nu0 + nn;
  const double shrink = beta_s > 0.0 ? beta0 * nn / beta_s : 0.0;
  for (int a = threadIdx.x; a < D; a += blockDim.x) {
    xbar[a] = n > 0 ? H[a] / nn : 0.0;
    dv[a] = mu0[a] - xbar[a];
  }
  __syncthreads();
  // W*^{-1} = W0^{-1} + (sum x x^T - n xbar xbar^T) + shrink dv dv^T (full matrix)
  for (int q = threadIdx.x; q < DD; q += blockDim.x) {
    const int i = q / D, j = q % D;
    const int a = min(i, j), e = max(i, j);
    const double sxx = H[D + a * D - a * (a - 1) / 2 + (e - a)];
    A[q] = W0inv[q] + (sxx - nn * xbar[i] * xbar[j]) + shrink * dv[i] * dv[j];
  }
  __syncthreads();
  for (int a = threadIdx.x; a < D; a += blockDim.x)
    xbar[a] = (beta0 * mu0[a] + nn * xbar[a]) / beta_s;  // mu0*
  // W* = R^{-T} R^{-1}, F = chol(W*)
  blk_cholesky(A, D, &bad);
  blk_lower_inverse(A, B, D);
  for (int q = threadIdx.x; q < DD; q += blockDim.x) {
    const int i = q / D, j = q % D;
    double t = 0.0;
    for (int m = max(i, j); m < D; ++m) t += B[m * D + i] * B[m * D + j];
    C[q] = t;
  }
  __syncthreads();
  blk_cholesky(C, D, &bad);
  // E = F B with Bartlett's lower triangular B
  for (int q = threadIdx.x; q < DD; q += blockDim.x) {
    const int i = q / D, j = q % D;
    double t = 0.0;
    for (int m = j; m <= i; ++m) {
      const double bm = m == j ? sqrt(chi2[j]) : offd[(int64_t)m * (m - 1) / 2 + j];
      t += C[i * D + m] * bm;
    }
    E[q] = t;
  }
  __syncthreads();
  blk_mul_abt(E, E, Lam_out, D);
  for (int q = threadIdx.x; q < DD; q += blockDim.x) G[q] = beta_s * Lam_out[q];
  blk_cholesky(G, D, &bad);
  // mu = mu0* + R^{-T} zmu (back substitution, one thread)
  if (threadIdx.x == 0) {
    for (int i = D - 1; i >= 0; --i) {
      double t = zmu[i];
      for (int m = i + 1; m < D; ++m) t -= G[m * D + i] * tmp[m];
      tmp[i] = t / G[i * D + i];
    }
    for (int i = 0; i < D; ++i) mu_out[i] = xbar[i] + tmp[i];
    *status = bad ? 1 : 0;
  }
}

}  // namespace

hipError_t launch_prior_prepare(const double *Lam, const double *mu, int D, int DP, double alpha,
                                float *init, float *K, float *mu32, double *scratch, int32_t *ok,
                                hipStream_t s) {
  if (D < 1 || D > 128 || !(alpha > 0.0)) return hipErrorInvalidValue;
  const int LD = lane_width(D);
  const int aug_col = (!LD && ((D + 3) & ~3) < DP) ? ((D + 3) & ~3) : -1;
  hipLaunchKernelGGL(k_prior_prepare, dim3(1), dim3(kBayesBlock), 0, s, Lam, mu, D, DP, LD,
                     aug_col, alpha, init, K, mu32, scratch, ok);
  return hipGetLastError();
}

hipError_t launch_prior_rows(const int32_t *rows, int64_t n, int D, const float *K,
                             const float *mu32, const int32_t *ok, const float *z, float *X,
                             int32_t *flag, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_prior_rows, dim3((unsigned)((n + 63) / 64)), dim3(64), 0, s, rows, n, D, K,
                     mu32, ok, z, X, flag);
  return hipGetLastError();
}

int hyper_blocks(int64_t n) {
  return (int)std::max<int64_t>(1, std::min<int64_t>(kHyperBlocks, (n + kMomentRows - 1) / kMomentRows));
}

hipError_t launch_hyper_moments(const float *X, int64_t n, int D, double *partials, hipStream_t s) {
  if (D < 1 || D > 128) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_hyper_moments, dim3((unsigned)hyper_blocks(n)), dim3(kBayesBlock), 0, s, X,
                     n, D, partials);
  return hipGetLastError();
}

hipError_t launch_hyper_sample(const double *partials, int nblk, int64_t n, int D,
                               const double *mu0, double beta0, const double *W0inv, double nu0,
                               const double *chi2, const double *offd, const double *zmu,
                               double *scratch, double *mu_out, double *Lam_out, int32_t *status,
                               hipStream_t s) {
  if (D < 1 || D > 128) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_hyper_sample, dim3(1), dim3(kBayesBlock), 0, s, partials, nblk, n, D, mu0,
                     beta0, W0inv, nu0, chi2, offd, zmu, scratch, mu_out, Lam_out, status);
  return hipGetLastError();
}

}  // namespace als
