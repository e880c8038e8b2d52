// Internal declarations shared by the HIP translation units of libals.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace als {

// One unit of Gram work: a whole row, or one chunk of a split ("hub") row.
struct WorkItem {
  int64_t start;  // first rating of the item, offset into the side's idx/val arrays
  int64_t slot;   // workspace slot of the item's partial normal equations (batch local)
  int32_t len;    // ratings in the item
  int32_t row;    // solved-side row the item belongs to
};
static_assert(sizeof(WorkItem) == 24, "WorkItem layout");

// One row to solve. A row with nslots == 0 builds its normal equations from its
// ratings [start, start + deg); a split row sums nslots workspace slots.
struct RowTask {
  int64_t start;    // first rating of the row
  int64_t slot0;    // batch-local slot of the row's first chunk (split rows)
  int32_t row;
  int32_t deg;      // n_s, number of ratings of the row
  int32_t nslots;
  int32_t sse_idx;  // where the row's entering-state squared residuals go (-1: split row)
};
static_assert(sizeof(RowTask) == 32, "RowTask layout");

// The staged fixed side is addressed with 32-bit byte offsets:
// (rows + 1) * DP * 4 must stay below 2^32.
constexpr int64_t kMaxStagedBytes = (1LL << 32) - 1;

// Padded factor width: D rounded up to the 16-wide MFMA tile.
inline int padded_width(int D) { return ((D + 15) / 16) * 16; }
// Upper-triangle 16x16 tiles of a DP x DP Gram matrix.
constexpr int num_tiles(int dp) { return (dp / 16) * (dp / 16 + 1) / 2; }
// Floats per workspace slot: the tiles in MFMA register order, then the right-hand side.
constexpr size_t slot_floats(int dp) { return (size_t)num_tiles(dp) * 256 + (size_t)dp; }
inline size_t slot_floats_rt(int dp) { int t = dp / 16; return (size_t)(t * (t + 1) / 2) * 256 + dp; }

// Bayesian row prior of one Gibbs half-sweep (BPMF / BPTF): each row's system starts
// from Lambda / alpha (identity on the padding) and Lambda mu / alpha instead of
// lambda n_s I and 0, and zscale * z_s is added to the forward-substitution result, so
// that the solve returns the conditional draw mu* + L*^{-T} z_s. init == nullptr: ALS.
struct RowPrior {
  const float *init = nullptr;  // the row kernel: one workspace slot (tiles in MFMA register
                                // order, then the right-hand side); the one-lane solve: one
                                // packed record (upper triangle, then the right-hand side)
  const float *z = nullptr;     // standard normal variates, [rows of the side x D]
  float zscale = 0.f;           // 1 / sqrt(alpha)
  // The time chain of BPTF: row r's prior is scale * init (scale_last * init for row
  // last_row), plus the per-row right-hand side h0 [rows x D] (already divided by alpha)
  // when h0 is set. The matrix and tensor Gibbs draws keep scale = 1, no h0.
  float scale = 1.f;
  float scale_last = 1.f;
  int64_t last_row = -1;
  const float *h0 = nullptr;

  __host__ __device__ float scale_of(int64_t row) const {
    return row == last_row ? scale_last : scale;
  }
};

// Tensor ALS: the second index of every rating (aligned with idx / val) and the second
// staged table; a rating's fixed vector is the elementwise product Fp[idx] * Tp[idx2].
// idx2 == nullptr: the matrix case.
struct Hadamard {
  const int32_t *idx2 = nullptr;
  const float *Tp = nullptr;
};

// ---- launchers (each returns the launch's hipError_t) ----------------------------------

// Column-major copy of a CSR matrix, built on the device (layout.hip).
// scratch_cnt: int32[nblk * n_cols]; tot: int64[n_cols]; col_ptr: int64[n_cols + 1].
hipError_t launch_csc_build(const int64_t *row_ptr, const int32_t *col, const uint8_t *val,
                            int64_t n_rows, int64_t n_cols, int64_t rows_per_blk, int64_t nblk,
                            int32_t *scratch_cnt, int64_t *tot, int64_t *col_ptr,
                            int32_t *row_idx, uint8_t *val_t, hipStream_t s);

// The same transpose applied to a per-rating float array (weights): w_t[q] = w[p]
// where q is the CSC position of CSR entry p, with col_ptr from launch_csc_build.
// The position of (row, column) is col_ptr[column] plus the number of earlier rows
// in that column, whatever the row blocking, so it matches the build.
hipError_t launch_csc_permute_f32(const int64_t *row_ptr, const int32_t *col, const float *w,
                                  int64_t n_rows, int64_t n_cols, int64_t rows_per_blk,
                                  int64_t nblk, int32_t *scratch_cnt, int64_t *tot,
                                  const int64_t *col_ptr, float *w_t, hipStream_t s);

// Copy of the fixed factors [n x D] into a zero-padded [(n + 1) x DP] buffer whose
// row n is all zero (rowsolve.hip).
hipError_t launch_stage_fixed(const float *F, int64_t n, int D, int DP, float *Fp, hipStream_t s);

// Partial normal equations of the chunks of split rows, into their workspace
// slots, with the chunks' entering-state squared residuals (rowsolve.hip).
// wts (here and below): per-rating weights aligned with idx / val for weighted ALS,
// or null for plain ALS.
hipError_t launch_gram_chunks(int dp, const WorkItem *items, int64_t n, const int32_t *idx,
                              const uint8_t *val, const float *wts, const float *Fp,
                              int64_t n_fixed, const float *Xold, int D, float *ws, double *sse,
                              const Hadamard &hd, hipStream_t s);

// Fused per-row normal equations, regularisation, Cholesky and solves; X is read
// (entering state) and overwritten in place (rowsolve.hip).
// cyc_gram / cyc_solve: both null, or arrays of n_rows doubles that receive each
// row's wavefront clock cycles spent before the factorisation (gather, Gram and
// residuals, or the sum of chunk partials) and from there on (factorisation, solves,
// write); a measurement aid that leaves the results unchanged.
// pr: the Bayesian prior (Gibbs half-sweep) or a default RowPrior (ALS; lam is used).
hipError_t launch_rows(int dp, const RowTask *rows, int64_t n_rows, const int32_t *idx,
                       const uint8_t *val, const float *wts, const float *Fp, int64_t n_fixed,
                       const float *ws, int D, float lam, float *X, double *sse, int32_t *flag,
                       double *cyc_gram, double *cyc_solve, const RowPrior &pr,
                       const Hadamard &hd, hipStream_t s);

// Per-item sums of squared residuals with the rows of X against the staged
// fixed side Fp (row stride DP, n_fixed rows and the zero row) (residual.hip).
hipError_t launch_resid(int dp, const WorkItem *items, int64_t n_items, const int32_t *idx,
                        const uint8_t *val, const float *Fp, int64_t n_fixed, const float *X,
                        int D, double *sse_items, const Hadamard &hd, hipStream_t s);

// Widths solved one row per lane (registers hold the packed normal equations).
inline int lane_width(int D) { return D <= 16 ? 16 : (D <= 20 ? 20 : 0); }
// Floats of one row's packed normal equations: upper triangle, right-hand side,
// rounded up to a multiple of 4.
constexpr int ne_floats(int ld) { return ((ld * (ld + 1) / 2 + ld) + 3) / 4 * 4; }

// Gram of rows or chunks packed into normal-equation records (lanesolve.hip):
// items [0, n_chunk_items) write to ws at their slot, the rest to ne at their slot.
hipError_t launch_gram_ne(int D, const WorkItem *items, int64_t n_items, int64_t n_chunk_items,
                          const int32_t *idx, const uint8_t *val, const float *wts,
                          const float *Fp, int64_t n_fixed, const float *Xold, float *ws,
                          float *ne, double *sse, const Hadamard &hd, hipStream_t s);

// One row per lane: regularise, Cholesky, solve, write (lanesolve.hip). Row i of
// the launch uses record base + i; its first n_split rows are split rows whose
// chunk records (in ws) are summed into their records first.
hipError_t launch_solve_lane(int D, const RowTask *rows, int64_t n_rows, int64_t n_split,
                             int64_t base, const float *ws, float *ne, float lam, float *X,
                             int32_t *flag, const RowPrior &pr, hipStream_t s);

// Fixed-order sum of n doubles into *out; partials: double[reduce_partials(n)]. host_out, if
// given, is the device address of mapped, coherent pinned host memory that receives the total
// as well; flag and host_flag (both or neither) copy one device int32 to such memory.
int64_t reduce_partials(int64_t n);
hipError_t launch_reduce(const double *v, int64_t n, double *partials, double *out,
                         hipStream_t s, double *host_out = nullptr,
                         const int32_t *flag = nullptr, int32_t *host_flag = nullptr);

hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s);

// Packed upper triangle of an LD x LD matrix, row by row (one-lane solve records).
template <int LD>
__host__ __device__ constexpr int tri(int a, int b) {  // a <= b
  return a * LD - a * (a - 1) / 2 + (b - a);
}

// ---- Bayesian Gibbs step (bayes.hip) ----------------------------------------------------

// fp64 scratch (doubles) of the hyperparameter draw: the summed moments and 16 segment
// sums of them.
inline size_t bayes_scratch_doubles(int D) { return (size_t)17 * (D + D * (D + 1) / 2) + 8; }
// Floats of the prior image: a workspace slot (D > 20) or a packed record (D <= 20).
inline size_t prior_init_floats(int D, int DP) {
  return lane_width(D) ? (size_t)ne_floats(lane_width(D)) : slot_floats_rt(DP);
}

// Prior image of a Gibbs half-sweep from the device hyperparameters Lambda (D x D) and mu
// (fp64): init (prior_init_floats) and mu in fp32; with need_factor (the side has rows
// without ratings) also the lower Cholesky factor L of Lambda (fp32 D x D) and *ok = 1,
// or 0 when Lambda is not numerically SPD.
hipError_t launch_prior_prepare(const double *Lam, const double *mu, int D, int DP, double alpha,
                                bool need_factor, float *init, float *L, float *mu32, int32_t *ok,
                                hipStream_t s);
// Rows without ratings drawn from the prior: X[row] = mu + L^{-T} z_row (flagged when !*ok).
hipError_t launch_prior_rows(const int32_t *rows, int64_t n, int D, const float *L,
                             const float *mu32, const int32_t *ok, const float *z, float *X,
                             int32_t *flag, hipStream_t s);
// Per-block fp64 sums of x and of the upper triangle of x x^T over the n rows of X
// (n x D): hyper_blocks(n) blocks, hyper_entries(D) doubles each.
int hyper_blocks(int64_t n);
inline int hyper_entries(int D) { return D + D * (D + 1) / 2; }
hipError_t launch_hyper_moments(const float *X, int64_t n, int D, double *partials, hipStream_t s);
// Normal-Wishart posterior from the moments and a Bartlett draw of (mu, Lambda) from it,
// in fp64 on one workgroup; *status = 0, or 1 when a factorisation fails.
hipError_t launch_hyper_sample(const double *partials, int nblk, int64_t n, int D,
                               const double *mu0, double beta0, const double *W0inv, double nu0,
                               const double *chi2, const double *offd, const double *zmu,
                               double *scratch, double *mu_out, double *Lam_out, int32_t *status,
                               hipStream_t s);
// The time chain of BPTF: h0 (K x D, fp32) of the bins k = parity, parity + 2, ...:
// Lambda_T (m_k + [k < K - 1] T_{k+1}) / alpha with m_0 = mu_T and m_k = T_{k-1}.
hipError_t launch_time_rhs(const float *T, int64_t K, int D, const double *Lam, const double *mu,
                           double alpha, int parity, float *h0, hipStream_t s);
// The chain's Normal-Wishart posterior (the moments of T_0 as one row, plus the step
// scatter in extra, D (D + 1) / 2 doubles, summed over nblk slices of per steps each from
// step_partials, nblk x D (D + 1) / 2 doubles; time_step_blocks gives the split) and the
// Bartlett draw of (mu_T, Lambda_T).
void time_step_blocks(int64_t K, int D, int64_t &per, int64_t &nblk);
hipError_t launch_time_hyper(const float *T, int64_t K, int D, const double *mu0, double beta0,
                             const double *W0inv, double nu0, const double *chi2,
                             const double *offd, const double *zmu, double *scratch,
                             double *step_partials, double *extra, double *mu_out,
                             double *Lam_out, int32_t *status, hipStream_t s);

// Predictions u_{users[p]} . v_{items[p]} of n pairs (predict.hip). pred (nullable)
// receives them, NaN for a pair with an index outside [0, M) x [0, N). With
// sse_blocks non-null, r holds the pairs' ratings and block b of pair_blocks(n, D)
// writes the fp64 sum of (r - r_hat)^2 over its pairs to sse_blocks[b].
int64_t pair_blocks(int64_t n, int D);
hipError_t launch_predict(const float *U, const float *V, int64_t M, int64_t N, int D, int64_t n,
                          const int32_t *users, const int32_t *items, const uint8_t *r,
                          float *pred, double *sse_blocks, hipStream_t s);

}  // namespace als
