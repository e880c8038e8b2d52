/*
 * Seeded synthetic rating matrices for the ALS workloads.
 *
 * This file only manufactures inputs: sparsity patterns with prescribed
 * degrees, popularity-weighted column choice, and integer ratings on 0..100.
 * It contains none of the ALS arithmetic (no Gram, no solve, no residual) and
 * is shared, as bytes on disk or in memory, by the fp64 oracle and by the HIP
 * library alike.
 *
 * Determinism: every row draws from its own counter-based stream
 * (SplitMix64, Steele/Lea/Flood 2014, seeded from (seed, row)), so the output
 * does not depend on the number of OpenMP threads.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

/* ---- SplitMix64 -------------------------------------------------------- */
static inline uint64_t sm64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
static inline uint64_t sm64_next(uint64_t *s) {
  *s += 0x9E3779B97F4A7C15ull;
  return sm64_mix(*s);
}
static inline uint64_t stream_seed(uint64_t seed, uint64_t key) {
  return sm64_mix(seed ^ sm64_mix(key * 0xD1B54A32D192ED03ull + 0x8CB92BA72F3D8DD7ull));
}
/* uniform double in [0,1) with 53 random bits */
static inline double u01(uint64_t *s) { return (double)(sm64_next(s) >> 11) * (1.0 / 9007199254740992.0); }
/* uniform double in (0,1] */
static inline double u01_open0(uint64_t *s) { return ((double)(sm64_next(s) >> 11) + 1.0) * (1.0 / 9007199254740992.0); }

/* ---- Vose alias table ---------------------------------------------------- */
typedef struct {
  int64_t n;
  double *prob;
  int32_t *alias;
} alias_t;

static int alias_build(alias_t *t, int64_t n, const double *w) {
  t->n = n;
  t->prob = (double *)malloc(sizeof(double) * n);
  t->alias = (int32_t *)malloc(sizeof(int32_t) * n);
  int32_t *small = (int32_t *)malloc(sizeof(int32_t) * n);
  int32_t *large = (int32_t *)malloc(sizeof(int32_t) * n);
  double *p = (double *)malloc(sizeof(double) * n);
  if (!t->prob || !t->alias || !small || !large || !p) return -1;
  double sum = 0.0;
  for (int64_t i = 0; i < n; ++i) sum += w[i];
  int64_t ns = 0, nl = 0;
  for (int64_t i = 0; i < n; ++i) {
    p[i] = w[i] * (double)n / sum;
    if (p[i] < 1.0) small[ns++] = (int32_t)i; else large[nl++] = (int32_t)i;
  }
  while (ns > 0 && nl > 0) {
    int32_t s = small[--ns], l = large[--nl];
    t->prob[s] = p[s];
    t->alias[s] = l;
    p[l] = (p[l] + p[s]) - 1.0;
    if (p[l] < 1.0) small[ns++] = l; else large[nl++] = l;
  }
  while (nl > 0) { int32_t l = large[--nl]; t->prob[l] = 1.0; t->alias[l] = l; }
  while (ns > 0) { int32_t s = small[--ns]; t->prob[s] = 1.0; t->alias[s] = s; }
  free(small); free(large); free(p);
  return 0;
}
static void alias_free(alias_t *t) { free(t->prob); free(t->alias); }
static inline int32_t alias_draw(const alias_t *t, uint64_t *s) {
  uint64_t r = sm64_next(s);
  int64_t i = (int64_t)((r >> 32) * (uint64_t)t->n >> 32);
  double u = (double)(r & 0xFFFFFFFFull) * (1.0 / 4294967296.0);
  return u < t->prob[i] ? (int32_t)i : t->alias[i];
}

/* ---- small sorting helpers (sorted, distinct columns per row) ------------ */
static void isort_i32(int32_t *a, int64_t n) {
  for (int64_t i = 1; i < n; ++i) {
    int32_t v = a[i];
    int64_t j = i - 1;
    while (j >= 0 && a[j] > v) { a[j + 1] = a[j]; --j; }
    a[j + 1] = v;
  }
}
/* LSD radix sort of non-negative int32 values below 2^31, 4 passes of 8 bits
 * (passes whose digit is constant are skipped). tmp has room for n values. */
static void rsort_i32(int32_t *a, int32_t *tmp, int64_t n) {
  if (n < 64) { isort_i32(a, n); return; }
  int32_t mx = 0;
  for (int64_t i = 0; i < n; ++i) if (a[i] > mx) mx = a[i];
  int32_t *src = a, *dst = tmp;
  for (int shift = 0; shift < 32 && (mx >> shift) != 0; shift += 8) {
    int64_t cnt[257];
    memset(cnt, 0, sizeof(cnt));
    for (int64_t i = 0; i < n; ++i) cnt[((src[i] >> shift) & 255) + 1]++;
    for (int b = 0; b < 256; ++b) cnt[b + 1] += cnt[b];
    for (int64_t i = 0; i < n; ++i) dst[cnt[(src[i] >> shift) & 255]++] = src[i];
    int32_t *t = src; src = dst; dst = t;
  }
  if (src != a) memcpy(a, src, sizeof(int32_t) * n);
}
static int64_t uniq_sorted(int32_t *a, int64_t n) {
  if (n == 0) return 0;
  int64_t m = 1;
  for (int64_t i = 1; i < n; ++i) if (a[i] != a[m - 1]) a[m++] = a[i];
  return m;
}

/* Hoare quickselect: after return, keys[k] holds the k-th largest (0-based). */
static double select_kth_largest(double *v, int64_t n, int64_t k) {
  int64_t lo = 0, hi = n - 1;
  while (lo < hi) {
    double pivot = v[lo + (hi - lo) / 2];
    int64_t i = lo, j = hi;
    while (i <= j) {
      while (v[i] > pivot) ++i;
      while (v[j] < pivot) --j;
      if (i <= j) { double t = v[i]; v[i] = v[j]; v[j] = t; ++i; --j; }
    }
    if (k <= j) hi = j; else if (k >= i) lo = i; else return v[k];
  }
  return v[k];
}

/*
 * Draw, for every row r, deg(r) = row_ptr[r+1]-row_ptr[r] distinct columns out
 * of n_cols, each column j having popularity weight w[j] > 0, and write them in
 * ascending order to col_out[row_ptr[r] .. row_ptr[r+1]).
 *  - deg >= n_cols: every column.
 *  - deg > n_cols/16: Efraimidis-Spirakis weighted sampling without
 *    replacement (keep the deg largest keys log(u)/w).
 *  - otherwise: alias-table draws, duplicates rejected and redrawn.
 * Returns 0, or -1 on allocation failure / bad degree.
 */
int synth_sample_rows(int64_t n_rows, const int64_t *row_ptr, int64_t n_cols,
                      const double *w, uint64_t seed, int32_t *col_out) {
  alias_t t;
  if (alias_build(&t, n_cols, w) != 0) return -1;
  int err = 0;
#pragma omp parallel
  {
    int32_t *buf = NULL, *tmp = NULL;
    double *keys = NULL, *keys2 = NULL;
    int64_t cap = 0;
#pragma omp for schedule(dynamic, 64)
    for (int64_t r = 0; r < n_rows; ++r) {
      int64_t d = row_ptr[r + 1] - row_ptr[r];
      int32_t *out = col_out + row_ptr[r];
      if (d <= 0) { if (d < 0) err = 1; continue; }
      if (d > n_cols) { err = 1; continue; }
      uint64_t s = stream_seed(seed, (uint64_t)r);
      if (d == n_cols) {
        for (int64_t j = 0; j < n_cols; ++j) out[j] = (int32_t)j;
        continue;
      }
      if (d * 16 > n_cols) {
        if (!keys) {
          keys = (double *)malloc(sizeof(double) * n_cols);
          keys2 = (double *)malloc(sizeof(double) * n_cols);
        }
        for (int64_t j = 0; j < n_cols; ++j) keys[j] = log(u01_open0(&s)) / w[j];
        memcpy(keys2, keys, sizeof(double) * n_cols);
        double thr = select_kth_largest(keys2, n_cols, d - 1);
        int64_t greater = 0;
        for (int64_t j = 0; j < n_cols; ++j) greater += keys[j] > thr;
        int64_t need_eq = d - greater, m = 0;
        for (int64_t j = 0; j < n_cols && m < d; ++j) {
          if (keys[j] > thr) out[m++] = (int32_t)j;
          else if (keys[j] == thr && need_eq > 0) { out[m++] = (int32_t)j; --need_eq; }
        }
        continue;
      }
      if (2 * d > cap) {
        free(buf); free(tmp);
        cap = 2 * d;
        buf = (int32_t *)malloc(sizeof(int32_t) * cap);
        tmp = (int32_t *)malloc(sizeof(int32_t) * cap);
      }
      int64_t have = 0;
      while (have < d) {
        int64_t want = d - have;
        for (int64_t k = 0; k < want; ++k) buf[have + k] = alias_draw(&t, &s);
        int64_t m = have + want;
        rsort_i32(buf, tmp, m);
        have = uniq_sorted(buf, m);
      }
      memcpy(out, buf, sizeof(int32_t) * d);
    }
    free(buf); free(tmp); free(keys); free(keys2);
  }
  alias_free(&t);
  return err ? -1 : 0;
}

/*
 * Rating mixture with no low-rank structure: per stored position p,
 * 30 % -> 0, 20 % -> uniform on 90..100, 50 % -> uniform on 1..89.
 */
void synth_ratings_mixture(int64_t nnz, uint64_t seed, uint8_t *val_out) {
  const int64_t block = 1 << 16;
  int64_t nb = (nnz + block - 1) / block;
#pragma omp parallel for schedule(static)
  for (int64_t b = 0; b < nb; ++b) {
    uint64_t s = stream_seed(seed, (uint64_t)b);
    int64_t e = (b + 1) * block < nnz ? (b + 1) * block : nnz;
    for (int64_t p = b * block; p < e; ++p) {
      uint64_t r = sm64_next(&s);
      uint32_t cls = (uint32_t)((r >> 32) % 10u);
      uint32_t v = (uint32_t)(r & 0xFFFFFFFFu);
      uint8_t out;
      if (cls < 3) out = 0;
      else if (cls < 5) out = (uint8_t)(90 + v % 11u);
      else out = (uint8_t)(1 + v % 89u);
      val_out[p] = out;
    }
  }
}

/*
 * Low-rank ground truth scores: score[p] = sum_k A[row(p), k] * B[col(p), k]
 * for every stored position p of the CSR pattern (A: n_rows x K, B: n_cols x K,
 * row-major fp64). Used only to give the synthetic ratings latent structure.
 */
void synth_lowrank_scores(int64_t n_rows, const int64_t *row_ptr, const int32_t *col,
                          int32_t K, const double *A, const double *B, double *score) {
#pragma omp parallel for schedule(dynamic, 256)
  for (int64_t r = 0; r < n_rows; ++r) {
    const double *a = A + (int64_t)K * r;
    for (int64_t p = row_ptr[r]; p < row_ptr[r + 1]; ++p) {
      const double *b = B + (int64_t)K * col[p];
      double acc = 0.0;
      for (int32_t k = 0; k < K; ++k) acc += a[k] * b[k];
      score[p] = acc;
    }
  }
}

/*
 * Quantise standardised scores to integer ratings:
 * val = clip(rint(mean_out + sd_out * (score - mu) / sigma + noise_sd * z), 0, 100)
 * with z ~ N(0,1) from a per-block stream (Box-Muller).
 */
void synth_quantise(int64_t nnz, const double *score, double mu, double sigma,
                    double mean_out, double sd_out, double noise_sd, uint64_t seed,
                    uint8_t *val_out) {
  const int64_t block = 1 << 16;
  int64_t nb = (nnz + block - 1) / block;
  const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for schedule(static)
  for (int64_t b = 0; b < nb; ++b) {
    uint64_t s = stream_seed(seed, (uint64_t)b);
    int64_t e = (b + 1) * block < nnz ? (b + 1) * block : nnz;
    for (int64_t p = b * block; p < e; ++p) {
      double u1 = u01_open0(&s), u2 = u01(&s);
      double z = sqrt(-2.0 * log(u1)) * cos(two_pi * u2);
      double x = mean_out + sd_out * (score[p] - mu) / sigma + noise_sd * z;
      x = rint(x);
      if (x < 0.0) x = 0.0;
      if (x > 100.0) x = 100.0;
      val_out[p] = (uint8_t)x;
    }
  }
}

/*
 * Stable counting transpose of a compressed pattern (used to turn an
 * item-major sample into user-major CSR). out_ptr has n_cols+1 entries.
 */
int synth_transpose(int64_t n_rows, int64_t n_cols, const int64_t *ptr, const int32_t *idx,
                    const uint8_t *val, int64_t *out_ptr, int32_t *out_idx, uint8_t *out_val) {
  memset(out_ptr, 0, sizeof(int64_t) * (n_cols + 1));
  int64_t nnz = ptr[n_rows];
  for (int64_t p = 0; p < nnz; ++p) out_ptr[idx[p] + 1]++;
  for (int64_t c = 0; c < n_cols; ++c) out_ptr[c + 1] += out_ptr[c];
  int64_t *cur = (int64_t *)malloc(sizeof(int64_t) * n_cols);
  if (!cur) return -1;
  memcpy(cur, out_ptr, sizeof(int64_t) * n_cols);
  for (int64_t r = 0; r < n_rows; ++r)
    for (int64_t p = ptr[r]; p < ptr[r + 1]; ++p) {
      int64_t q = cur[idx[p]]++;
      out_idx[q] = (int32_t)r;
      out_val[q] = val[p];
    }
  free(cur);
  return 0;
}
