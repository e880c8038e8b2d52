// Bayesian factorisation (BPTF, Sec. 2.2, which pairs the least-squares update with draws
// of the factor priors' parameters), in the form of the published BPMF / BPTF Gibbs sampler.
// Ratings are Gaussian with precision alpha around u . v; each row of a side has the
// prior N(mu, Lambda^{-1}); (mu, Lambda) has a Normal-Wishart hyperprior. The row draws
// reuse the half-sweep kernels (their BAYES variants): this file holds the rest.
//
//   k_prior_prepare   one workgroup, fp64: the prior image the row kernels start from
//                     (Lambda / alpha with the identity on the padding, and
//                     Lambda mu / alpha), laid out as a workspace slot (D > 20) or a
//                     packed record (D <= 20); and, when the side has rows without
//                     ratings, the Cholesky factor L of Lambda for them.
//   k_prior_rows      one lane per row without ratings: x = mu + L^{-T} z.
//   k_hyper_moments   per-block fp64 sums of x and of the upper triangle of x x^T over
//                     the side's rows (rows staged through LDS); products of two fp32
//                     values are exact in fp64, so only the summation order rounds.
//   k_hyper_reduce    the per-block partials summed in 16 fixed segments, in order.
//   k_hyper_sample    one workgroup, fp64: adds the segments in order, forms the
//                     Normal-Wishart posterior (beta* = beta0 + n, nu* = nu0 + n,
//                     mu0* = (beta0 mu0 + n xbar) / beta*, W*^{-1} = W0^{-1} + S +
//                     beta0 n / beta* (mu0 - xbar)(mu0 - xbar)^T with S the scatter
//                     about the mean), then Bartlett's draw: W* = F F^T, B lower
//                     triangular with B_ii = sqrt(chi2_i) and normal B_ij, Lambda =
//                     (F B)(F B)^T, and mu = mu0* + R^{-T} zmu with beta* Lambda = R R^T.
// The time chain of BPTF (T_0 ~ N(mu_T, Lambda_T^{-1}), T_k ~ N(T_{k-1}, Lambda_T^{-1})):
//   k_time_rhs        a bin's prior right-hand side Lambda_T (m_k + [k < K - 1] T_{k+1}) /
//                     alpha (m_k = mu_T for the first bin, else T_{k-1}) for the bins of
//                     one parity, in fp64; the bins of a parity are drawn together given
//                     the other parity.
//   k_time_moments    the moments of T_0 alone (n = 1), in the segment layout
//                     k_hyper_sample reads;
//   k_time_steps      the chain's step scatter sum_{k>=1} (T_k - T_{k-1})(T_k - T_{k-1})^T
//                     over a slice of the chain per block (the slice's bins staged in
//                     LDS, differences formed in fp64, exact for fp32 inputs), and
//   k_time_steps_sum  the slices added in order; k_hyper_sample adds the result to
//                     W*^{-1}.
// The variates (chi-square, normals) are inputs. Matrices live as fp64
// packed triangles in LDS (two of them, 132 KB at D = 128); the factorisations are
// right-looking Cholesky steps with a barrier between steps.
#include "internal.h"

namespace als {

namespace {

constexpr int kBayesBlock = 256;
constexpr int kStageFloats = 16384;  // LDS stage of the moment kernel (64 KB of rows)
constexpr int kHyperBlocks = 1024;
constexpr int kReduceSegs = 16;      // the moment partials are summed in 16 segments
constexpr int kMaxD = 128;
constexpr int kStepBlocks = 64;          // slices of the time chain's step scatter
constexpr int kStepStageFloats = 15360;  // LDS stage of a slice (60 KB)
constexpr int kPacked = kMaxD * (kMaxD + 1) / 2;
// 4 x 4 tiles of the upper block triangle of x x^T, per thread at most this many
constexpr int kTilesPerThread = ((kMaxD / 4) * (kMaxD / 4 + 1) / 2 + kBayesBlock - 1) / kBayesBlock;

// Index of (i, j), j <= i, in a packed lower triangle.
__device__ __forceinline__ int pl(int i, int j) { return i * (i + 1) / 2 + j; }

// In-place lower Cholesky factor of the packed lower triangle P (in LDS), right-looking:
// per column, the pivot's square root, the column scaled, then the trailing triangle
// updated, with barriers between. *bad is set when a pivot is not positive and finite
// (the step then continues with a unit pivot, so that every value stays defined).
__device__ void lds_cholesky(double *P, int D, int *bad) {
  for (int k = 0; k < D; ++k) {
    __syncthreads();
    const double p = P[pl(k, k)];
    const bool ok = p > 0.0 && isfinite(p);
    const double l = ok ? sqrt(p) : 1.0;
    if (!ok && threadIdx.x == 0) *bad = 1;
    __syncthreads();
    if (threadIdx.x == 0) P[pl(k, k)] = l;
    for (int i = k + 1 + threadIdx.x; i < D; i += blockDim.x) P[pl(i, k)] /= l;
    __syncthreads();
    // trailing triangle k < j <= i < D on a 16 x 16 grid of threads
    for (int i = k + 1 + (int)(threadIdx.x >> 4); i < D; i += 16) {
      const double lik = P[pl(i, k)];
      for (int j = k + 1 + (int)(threadIdx.x & 15); j <= i; j += 16)
        P[pl(i, j)] -= lik * P[pl(j, k)];
    }
  }
  __syncthreads();
}

// Li = L^{-1} for the packed lower triangles L and Li (in LDS), one column per thread
// (each column's forward substitution only reads L and its own earlier entries).
__device__ void lds_lower_inverse(const double *L, double *Li, int D) {
  for (int e = threadIdx.x; e < D; e += blockDim.x) {
    for (int i = e; i < D; ++i) {
      double s = i == e ? 1.0 : 0.0;
      for (int m = e; m < i; ++m) s -= L[pl(i, m)] * Li[pl(m, e)];
      Li[pl(i, e)] = s / L[pl(i, i)];
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(kBayesBlock) void k_prior_prepare(
    const double *__restrict__ Lam, const double *__restrict__ mu, int D, int DP, int LD,
    int aug_col, double alpha, int need_factor, float *__restrict__ init,
    float *__restrict__ K, float *__restrict__ mu32, int32_t *__restrict__ ok) {
  __shared__ double P1[kPacked];
  __shared__ double c[kMaxD];  // Lambda mu / alpha
  __shared__ int bad;
  if (threadIdx.x == 0) bad = 0;
  __shared__ double mus[kMaxD];
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    mus[d] = mu[d];
    mu32[d] = (float)mu[d];
  }
  // the lower triangle of Lambda (symmetric by contract) into LDS
  for (int i = (int)(threadIdx.x >> 4); i < D; i += 16)
    for (int j = (int)(threadIdx.x & 15); j <= i; j += 16) P1[pl(i, j)] = Lam[i * D + j];
  __syncthreads();
  auto lam = [&](int a, int b) -> double { return a >= b ? P1[pl(a, b)] : P1[pl(b, a)]; };
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    double t = 0.0;
    for (int e = 0; e < D; ++e) t += lam(d, e) * mus[e];
    c[d] = t / alpha;
  }
  __syncthreads();
  // entry (r, col) of the scaled prior matrix, the identity on the padding, and with the
  // augmented column (D > 20 only) holding Lambda mu / alpha
  auto entry = [&](int r, int col) -> float {
    if (r < D && col < D) return (float)(lam(r, col) / alpha);
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
  // the Cholesky factor L of Lambda for the rows without ratings, when the side has any
  // (the image is written above, so P1 can be factored in place)
  if (need_factor) {
    lds_cholesky(P1, D, &bad);
    for (int q = threadIdx.x; q < D * D; q += blockDim.x) {
      const int i = q / D, j = q % D;
      K[q] = j <= i ? (float)P1[pl(i, j)] : 0.f;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) *ok = bad ? 0 : 1;
}

__global__ __launch_bounds__(64) void k_prior_rows(const int32_t *__restrict__ rows, int64_t n,
                                                  int D, const float *__restrict__ L,
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
  // x = mu + L^{-T} z: back substitution with L^T into the row, then the mean added
  const float *__restrict__ zr = z + row * D;
  float *__restrict__ xr = X + row * D;
  for (int a = D - 1; a >= 0; --a) {
    float t = zr[a];
    for (int e = a + 1; e < D; ++e) t = fmaf(-L[e * D + a], xr[e], t);
    xr[a] = t / L[a * D + a];
  }
  for (int a = 0; a < D; ++a) xr[a] += mu32[a];
}

// Moments: the block's rows are staged through LDS; each thread accumulates whole 4 x 4
// tiles (I, J), I <= J, of the upper block triangle of x x^T (four values of each row
// feed sixteen products), and thread a < D the sum of feature a. When there are fewer
// tiles than threads, G = 256 / tiles threads share a tile, thread g of them taking the
// staged rows r = g mod G; their partial tiles are added in order of g at the end.
// Entries are written in the packed order: the D sums of x_a, then the upper triangle of
// x x^T row by row.
__global__ __launch_bounds__(kBayesBlock) void k_hyper_moments(const float *__restrict__ X,
                                                               int64_t n, int D,
                                                               double *__restrict__ partials) {
  __shared__ __align__(16) float xs_flat[kStageFloats];
  const int nb = (D + 3) / 4;       // 4-wide feature blocks
  const int w4 = 4 * nb;            // staged row width
  const int stage_rows = min(256, kStageFloats / w4);
  const int ntl = nb * (nb + 1) / 2;
  const int ne = D + D * (D + 1) / 2;
  const int G = max(1, kBayesBlock / ntl);  // threads per tile
  const int g = (int)threadIdx.x % G, slot = (int)threadIdx.x / G, slots = kBayesBlock / G;
  int ti[kTilesPerThread], tj[kTilesPerThread];
  double acc[kTilesPerThread][16], sx = 0.0;
#pragma unroll
  for (int k = 0; k < kTilesPerThread; ++k) {
    int t = slot + k * slots, I = 0;
    ti[k] = -1;
    tj[k] = -1;
    if (slot < slots && t < ntl) {
      while (t >= nb - I) {
        t -= nb - I;
        ++I;
      }
      ti[k] = I;
      tj[k] = I + t;
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[k][q] = 0.0;
  }
  const int64_t per = (n + gridDim.x - 1) / gridDim.x;
  const int64_t r0 = (int64_t)blockIdx.x * per, r1 = min(n, r0 + per);
  for (int64_t base = r0; base < r1; base += stage_rows) {
    const int rows = (int)min<int64_t>(stage_rows, r1 - base);
    __syncthreads();
    for (int q = threadIdx.x; q < rows * w4; q += kBayesBlock) {
      const int r = q / w4, d = q % w4;
      xs_flat[q] = d < D ? X[(base + r) * D + d] : 0.f;
    }
    __syncthreads();
    if ((int)threadIdx.x < D) {
      for (int r = 0; r < rows; ++r) sx += (double)xs_flat[r * w4 + threadIdx.x];
    }
#pragma unroll
    for (int k = 0; k < kTilesPerThread; ++k) {
      if (ti[k] >= 0) {
        const int a0 = 4 * ti[k], e0 = 4 * tj[k];
        for (int r = g; r < rows; r += G) {
          const float4 va = *reinterpret_cast<const float4 *>(xs_flat + r * w4 + a0);
          const float4 ve = *reinterpret_cast<const float4 *>(xs_flat + r * w4 + e0);
          const double xa[4] = {va.x, va.y, va.z, va.w};
          const double xe[4] = {ve.x, ve.y, ve.z, ve.w};
#pragma unroll
          for (int q = 0; q < 4; ++q) {
#pragma unroll
            for (int w = 0; w < 4; ++w) acc[k][4 * q + w] = fma(xa[q], xe[w], acc[k][4 * q + w]);
          }
        }
      }
    }
  }
  double *__restrict__ out = partials + (int64_t)blockIdx.x * ne;
  if ((int)threadIdx.x < D) out[threadIdx.x] = sx;
  // the G partial tiles of a slot are added in order of g through LDS (G > 1 means one
  // tile per thread)
  double *red = reinterpret_cast<double *>(xs_flat);  // 256 x 16 doubles = 32 KB
#pragma unroll
  for (int k = 0; k < kTilesPerThread; ++k) {
    if (G > 1) {
      __syncthreads();
#pragma unroll
      for (int q = 0; q < 16; ++q) red[threadIdx.x * 16 + q] = acc[k][q];
      __syncthreads();
      if (g == 0 && ti[k] >= 0) {
        for (int h = 1; h < G; ++h) {
#pragma unroll
          for (int q = 0; q < 16; ++q) acc[k][q] += red[(threadIdx.x + h) * 16 + q];
        }
      }
    }
    if (g == 0 && ti[k] >= 0) {
      const int a0 = 4 * ti[k], e0 = 4 * tj[k];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const int a = a0 + q, e = e0 + w;
          if (a <= e && e < D) out[D + a * D - a * (a - 1) / 2 + (e - a)] = acc[k][4 * q + w];
        }
      }
    }
  }
}

// Segment sums of the moment partials: thread (q, seg) adds entry q of the blocks of
// segment seg in block order (the loads of one thread are independent, so many are in
// flight); the draw kernel adds the segments in order.
__global__ __launch_bounds__(64) void k_hyper_reduce(const double *__restrict__ partials, int nblk,
                                                     int ne, double *__restrict__ seg_sums) {
  const int q = blockIdx.x * 64 + threadIdx.x;
  const int seg = blockIdx.y;
  if (q >= ne) return;
  const int per = (nblk + kReduceSegs - 1) / kReduceSegs;
  const int b0 = seg * per, b1 = min(nblk, b0 + per);
  double t = 0.0;
#pragma unroll 16
  for (int b = b0; b < b1; ++b) t += partials[(int64_t)b * ne + q];
  seg_sums[(int64_t)seg * ne + q] = t;
}

// Normal-Wishart posterior and Bartlett draw on two packed triangles in LDS:
//   P1 = W*^{-1} -> R (Cholesky);  P2 = R^{-1};  P1 = W* = R^{-T} R^{-1} -> F (Cholesky);
//   P2 = F B (lower times lower is lower);  P1 = Lambda = (F B)(F B)^T, written out;
//   P1 = beta* Lambda -> its Cholesky factor;  mu = mu0* + R^{-T} zmu.
// extra (nullable): a packed upper triangle added to W*^{-1} (the time chain's steps).
__global__ __launch_bounds__(kBayesBlock) void k_hyper_sample(
    const double *__restrict__ seg_sums, int64_t n, int D,
    const double *__restrict__ mu0, double beta0, const double *__restrict__ W0inv, double nu0,
    const double *__restrict__ chi2, const double *__restrict__ offd,
    const double *__restrict__ zmu, const double *__restrict__ extra, double *__restrict__ H,
    double *__restrict__ mu_out, double *__restrict__ Lam_out, int32_t *__restrict__ status) {
  __shared__ double P1[kPacked], P2[kPacked];
  __shared__ double xbar[kMaxD], dv[kMaxD], tmp[kMaxD];
  __shared__ int bad;
  if (threadIdx.x == 0) bad = 0;
  const int ne = D + D * (D + 1) / 2;
  // the moments: segment sums added in segment order (H: global scratch of ne doubles)
  for (int q = threadIdx.x; q < ne; q += blockDim.x) {
    double t = 0.0;
#pragma unroll
    for (int g = 0; g < kReduceSegs; ++g) t += seg_sums[(int64_t)g * ne + q];
    H[q] = t;
  }
  __syncthreads();
  const double nn = (double)n;
  const double beta_s = beta0 + nn;
  const double shrink = beta_s > 0.0 ? beta0 * nn / beta_s : 0.0;
  for (int a = threadIdx.x; a < D; a += blockDim.x) {
    xbar[a] = n > 0 ? H[a] / nn : 0.0;
    dv[a] = mu0[a] - xbar[a];
  }
  __syncthreads();
  // W*^{-1} = W0^{-1} + (sum x x^T - n xbar xbar^T) + shrink dv dv^T (lower triangle)
  for (int i = (int)(threadIdx.x >> 4); i < D; i += 16) {
    for (int j = (int)(threadIdx.x & 15); j <= i; j += 16) {
      const int q = j * D - j * (j - 1) / 2 + (i - j);
      const double sxx = H[D + q];
      P1[pl(i, j)] = W0inv[i * D + j] + (sxx - nn * xbar[i] * xbar[j]) + shrink * dv[i] * dv[j] +
                     (extra ? extra[q] : 0.0);
    }
  }
  __syncthreads();
  for (int a = threadIdx.x; a < D; a += blockDim.x)
    xbar[a] = (beta0 * mu0[a] + nn * xbar[a]) / beta_s;  // mu0*
  lds_cholesky(P1, D, &bad);
  lds_lower_inverse(P1, P2, D);
  // W* = R^{-T} R^{-1}: entry (i, j), j <= i, sums over m >= i
  for (int i = (int)(threadIdx.x >> 4); i < D; i += 16) {
    for (int j = (int)(threadIdx.x & 15); j <= i; j += 16) {
      double t = 0.0;
      for (int m = i; m < D; ++m) t += P2[pl(m, i)] * P2[pl(m, j)];
      P1[pl(i, j)] = t;
    }
  }
  lds_cholesky(P1, D, &bad);  // F
  // Bartlett's B into P2 (packed in the same order: row m, column j < m: offd[pl(m, j) - m])
  for (int q = threadIdx.x; q < D * (D + 1) / 2; q += blockDim.x) {
    int m = (int)((sqrt(8.0 * q + 1.0) - 1.0) * 0.5);
    while (pl(m, 0) > q) --m;
    while (pl(m + 1, 0) <= q) ++m;
    const int j = q - pl(m, 0);
    P2[q] = j == m ? sqrt(chi2[m]) : offd[q - m];
  }
  __syncthreads();
  // E = F B in place of F, one row per thread: entry (i, j) needs F[i][m] for m >= j only,
  // so a row is overwritten in increasing j
  for (int i = threadIdx.x; i < D; i += blockDim.x) {
    for (int j = 0; j <= i; ++j) {
      double t = 0.0;
      for (int m = j; m <= i; ++m) t += P1[pl(i, m)] * P2[pl(m, j)];
      P1[pl(i, j)] = t;
    }
  }
  __syncthreads();
  // Lambda = E E^T into P2
  for (int i = (int)(threadIdx.x >> 4); i < D; i += 16) {
    for (int j = (int)(threadIdx.x & 15); j <= i; j += 16) {
      double t = 0.0;
      for (int m = 0; m <= j; ++m) t += P1[pl(i, m)] * P1[pl(j, m)];
      P2[pl(i, j)] = t;
      Lam_out[i * D + j] = t;
      Lam_out[j * D + i] = t;
    }
  }
  __syncthreads();
  for (int q = threadIdx.x; q < D * (D + 1) / 2; q += blockDim.x) P2[q] *= beta_s;
  lds_cholesky(P2, D, &bad);
  // mu = mu0* + R^{-T} zmu: back substitution with R^T, column by column (tmp holds the
  // right-hand side still to be reduced)
  for (int i = threadIdx.x; i < D; i += blockDim.x) tmp[i] = zmu[i];
  for (int i = D - 1; i >= 0; --i) {
    __syncthreads();
    const double ti = tmp[i] / P2[pl(i, i)];
    __syncthreads();
    if (threadIdx.x == 0) tmp[i] = ti;
    for (int m = threadIdx.x; m < i; m += blockDim.x) tmp[m] -= P2[pl(i, m)] * ti;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < D; i += blockDim.x) mu_out[i] = xbar[i] + tmp[i];
  if (threadIdx.x == 0) *status = bad ? 1 : 0;
}

// Row a and column b (a <= b) of packed upper-triangle entry t (rows in order).
__device__ inline void upper_entry(int t, int D, int &a, int &b) {
  a = 0;
  while (t >= D - a) {
    t -= D - a;
    ++a;
  }
  b = a + t;
}

__global__ __launch_bounds__(256) void k_time_rhs(const float *__restrict__ T, int64_t K, int D,
                                                  const double *__restrict__ Lam,
                                                  const double *__restrict__ mu, double inv_alpha,
                                                  int parity, float *__restrict__ h0) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t nk = (K - parity + 1) / 2;  // bins of this parity
  if (t >= nk * D) return;
  const int64_t k = parity + 2 * (t / D);
  const int a = (int)(t % D);
  double acc = 0.0;
  for (int e = 0; e < D; ++e) {
    const double prev = k == 0 ? mu[e] : (double)T[(k - 1) * D + e];
    const double next = k < K - 1 ? (double)T[(k + 1) * D + e] : 0.0;
    acc += Lam[a * D + e] * (prev + next);
  }
  h0[k * D + a] = (float)(acc * inv_alpha);
}

__global__ __launch_bounds__(256) void k_time_moments(const float *__restrict__ T, int D,
                                                      double *__restrict__ seg_sums) {
  const int ne = D + D * (D + 1) / 2;
  for (int q = blockIdx.x * 256 + threadIdx.x; q < kReduceSegs * ne; q += gridDim.x * 256) {
    const int g = q / ne, e = q % ne;
    double v = 0.0;
    if (g == 0) {
      if (e < D) {
        v = (double)T[e];
      } else {
        int a, b;
        upper_entry(e - D, D, a, b);
        v = (double)T[a] * (double)T[b];
      }
    }
    seg_sums[q] = v;
  }
}

// Block b takes the steps k = 1 + b per .. min(K, 1 + (b + 1) per) - 1, with the bins
// k - 1 .. of its slice staged in LDS (dynamic, (per + 1) D floats).
__global__ __launch_bounds__(256) void k_time_steps(const float *__restrict__ T, int64_t K, int D,
                                                    int64_t per, double *__restrict__ partials) {
  extern __shared__ float rows[];
  const int ntri = D * (D + 1) / 2;
  const int64_t k0 = 1 + (int64_t)blockIdx.x * per;
  const int64_t k1 = min(K, k0 + per);
  double *__restrict__ out = partials + (int64_t)blockIdx.x * ntri;
  const int nr = k0 < K ? (int)(k1 - k0 + 1) : 0;  // bins k0 - 1 .. k1 - 1
  for (int q = threadIdx.x; q < nr * D; q += 256) rows[q] = T[(k0 - 1) * D + q];
  __syncthreads();
  for (int q = threadIdx.x; q < ntri; q += 256) {
    int a, b;
    upper_entry(q, D, a, b);
    double acc = 0.0;
    for (int r = 1; r < nr; ++r)
      acc += ((double)rows[r * D + a] - (double)rows[(r - 1) * D + a]) *
             ((double)rows[r * D + b] - (double)rows[(r - 1) * D + b]);
    out[q] = acc;
  }
}

__global__ __launch_bounds__(256) void k_time_steps_sum(const double *__restrict__ partials,
                                                        int nblk, int ntri,
                                                        double *__restrict__ extra) {
  const int q = blockIdx.x * 256 + threadIdx.x;
  if (q >= ntri) return;
  double t = 0.0;
  for (int b = 0; b < nblk; ++b) t += partials[(int64_t)b * ntri + q];
  extra[q] = t;
}

}  // namespace

hipError_t launch_prior_prepare(const double *Lam, const double *mu, int D, int DP, double alpha,
                                bool need_factor, float *init, float *L, float *mu32, int32_t *ok,
                                hipStream_t s) {
  if (D < 1 || D > 128 || !(alpha > 0.0)) return hipErrorInvalidValue;
  const int LD = lane_width(D);
  const int aug_col = (!LD && ((D + 3) & ~3) < DP) ? ((D + 3) & ~3) : -1;
  hipLaunchKernelGGL(k_prior_prepare, dim3(1), dim3(kBayesBlock), 0, s, Lam, mu, D, DP, LD,
                     aug_col, alpha, need_factor ? 1 : 0, init, L, mu32, ok);
  return hipGetLastError();
}

hipError_t launch_prior_rows(const int32_t *rows, int64_t n, int D, const float *L,
                             const float *mu32, const int32_t *ok, const float *z, float *X,
                             int32_t *flag, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_prior_rows, dim3((unsigned)((n + 63) / 64)), dim3(64), 0, s, rows, n, D, L,
                     mu32, ok, z, X, flag);
  return hipGetLastError();
}

int hyper_blocks(int64_t n) {
  return (int)std::max<int64_t>(1, std::min<int64_t>(kHyperBlocks, (n + 63) / 64));
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
  if (D < 1 || D > 128 || nblk < 1) return hipErrorInvalidValue;
  const int ne = hyper_entries(D);
  double *seg_sums = scratch + ne + 8;
  hipLaunchKernelGGL(k_hyper_reduce, dim3((unsigned)((ne + 63) / 64), kReduceSegs), dim3(64), 0, s,
                     partials, nblk, ne, seg_sums);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_hyper_sample, dim3(1), dim3(kBayesBlock), 0, s, seg_sums, n, D, mu0,
                     beta0, W0inv, nu0, chi2, offd, zmu, (const double *)nullptr, scratch, mu_out,
                     Lam_out, status);
  return hipGetLastError();
}

hipError_t launch_time_rhs(const float *T, int64_t K, int D, const double *Lam, const double *mu,
                           double alpha, int parity, float *h0, hipStream_t s) {
  if (D < 1 || D > 128 || K < 1 || (parity != 0 && parity != 1) || !(alpha > 0.0))
    return hipErrorInvalidValue;
  const int64_t threads = (K - parity + 1) / 2 * D;
  if (threads == 0) return hipSuccess;
  hipLaunchKernelGGL(k_time_rhs, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, T, K,
                     D, Lam, mu, 1.0 / alpha, parity, h0);
  return hipGetLastError();
}

void time_step_blocks(int64_t K, int D, int64_t &per, int64_t &nblk) {
  const int64_t steps = std::max<int64_t>(K - 1, 0);
  const int64_t max_rows = kStepStageFloats / D;  // staged bins per block
  per = std::max<int64_t>(1, std::min<int64_t>((steps + kStepBlocks - 1) / kStepBlocks,
                                               max_rows - 1));
  nblk = std::max<int64_t>(1, (steps + per - 1) / per);
}

hipError_t launch_time_hyper(const float *T, int64_t K, int D, const double *mu0, double beta0,
                             const double *W0inv, double nu0, const double *chi2,
                             const double *offd, const double *zmu, double *scratch,
                             double *step_partials, double *extra, double *mu_out,
                             double *Lam_out, int32_t *status, hipStream_t s) {
  if (D < 1 || D > 128 || K < 1) return hipErrorInvalidValue;
  const int ne = hyper_entries(D), ntri = D * (D + 1) / 2;
  double *seg_sums = scratch + ne + 8;
  hipLaunchKernelGGL(k_time_moments, dim3((unsigned)((kReduceSegs * ne + 255) / 256)), dim3(256),
                     0, s, T, D, seg_sums);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  int64_t per = 0, nblk = 0;
  time_step_blocks(K, D, per, nblk);
  hipLaunchKernelGGL(k_time_steps, dim3((unsigned)nblk), dim3(256),
                     (size_t)(per + 1) * D * sizeof(float), s, T, K, D, per, step_partials);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_time_steps_sum, dim3((unsigned)((ntri + 255) / 256)), dim3(256), 0, s,
                     step_partials, (int)nblk, ntri, extra);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_hyper_sample, dim3(1), dim3(kBayesBlock), 0, s, seg_sums, (int64_t)1, D,
                     mu0, beta0, W0inv, nu0, chi2, offd, zmu, (const double *)extra, scratch,
                     mu_out, Lam_out, status);
  return hipGetLastError();
}

}  // namespace als
