// Host side of libals: the C ABI declared in include/als.h.
//
// als_create validates the user-major CSR, copies it to the device, builds the
// item-major copy on the device (layout.hip) and plans both sides: rows with
// ratings are ordered by descending degree (largest work first); rows above
// the hub threshold are cut into fixed-size chunks whose partial normal
// equations go to workspace slots. A half-sweep stages the fixed side into a
// padded copy, then runs per batch the chunk kernel and the fused row kernel
// (rowsolve.hip), and reduces the entering-state squared residuals; the
// new-state RMSE is an extra residual pass (residual.hip), run on request.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "als.h"
#include "internal.h"

using als::RowTask;
using als::WorkItem;

namespace {

constexpr int32_t kDefaultHubThreshold = 8192;
constexpr int32_t kDefaultChunk = 4096;
constexpr int64_t kDefaultWorkspace = 48LL << 30;
// cap on the block-by-column count table of the device transpose
constexpr int64_t kCscTableEntries = 1LL << 29;

struct Batch {
  int64_t gitem_off;  // first gather item of the batch
  int64_t n_gchunks;  // its chunks of split rows (they come first)
  int64_t n_gitems;   // chunks + unsplit rows
  int64_t row_off, n_rows;
  int64_t n_split;    // the batch's first n_split rows are split rows
  int64_t n_slots;    // workspace slots used by the batch's chunks
};

struct SidePlan {
  int64_t n_rows = 0;       // rows of this side
  int64_t rows_with = 0;    // rows with at least one rating
  int64_t split_rows = 0;   // rows cut into chunks
  int64_t n_chunks = 0;
  int64_t max_deg = 0;
  int64_t max_slots = 0;    // largest batch, in slots
  std::vector<Batch> batches;
  std::vector<WorkItem> gitems;  // per batch: chunks of split rows, then unsplit rows
  std::vector<RowTask> rows;     // every row with ratings, batch-major, descending degree
  WorkItem *d_gitems = nullptr;
  RowTask *d_rows = nullptr;
  std::vector<int32_t> zero_rows;  // rows without ratings (drawn from the prior when Bayesian)
  int32_t *d_zero_rows = nullptr;
};

constexpr int kPhases = 5;  // stage, chunks, rows, residual, reduce

struct ProfEvent {
  int phase;
  hipEvent_t a, b;
};

}  // namespace

struct als_ctx {
  int64_t M = 0, N = 0, nnz = 0;
  int32_t D = 0, DP = 0;
  hipStream_t stream = nullptr;
  int device = 0;
  als_tuning tune{};
  std::vector<int64_t> h_row_ptr, h_col_ptr;
  int64_t *d_row_ptr = nullptr;
  int32_t *d_col = nullptr;
  uint8_t *d_val = nullptr;
  int64_t *d_col_ptr = nullptr;
  int32_t *d_row_idx = nullptr;
  uint8_t *d_val_t = nullptr;
  float *d_w = nullptr;    // weighted ALS: per-rating weights in CSR order (null: plain ALS)
  float *d_w_t = nullptr;  // the same weights in CSC order
  SidePlan plan[5];  // users, items, (tensor ALS) time bins, and the even / odd time bins
  float *d_ws = nullptr;
  size_t ws_bytes = 0;
  float *d_fpad = nullptr;       // staged fixed side [(max(M, N) + 1) x DP], last row zero
  float *d_ne = nullptr;         // packed normal equations, one record per row (narrow D)
  bool lane_solve = false;       // narrow D: Gram records + one row per lane solve
  double *d_sse_items = nullptr; // per chunk / row / piece squared residuals
  double *d_partials = nullptr;
  double *d_sse_in = nullptr;    // entering-state SSE of the last half-sweep
  double *d_sse_total = nullptr; // SSE of the last residual pass
  int32_t *d_flag = nullptr;
  double *h_sse = nullptr;    // pinned
  double *h_sse_in = nullptr; // pinned, mapped [2]: the entering-state SSE of the last
                              // half-sweep, in one part, or two for the time chain's even and
                              // odd passes
  int sse_in_parts = 1;
  int32_t *h_flag = nullptr;  // pinned, mapped
  double *hd_sse_in = nullptr; // device addresses of h_sse_in and h_flag
  int32_t *hd_flag = nullptr;
  int last_side = -1;
  std::string err;
  bool profiling = false;
  int prof_mode = 0;  // 1: every phase; 2: the launches that build the normal equations
  std::vector<ProfEvent> prof_pending;
  std::vector<hipEvent_t> ev_pool;
  double prof_ms[kPhases] = {0, 0, 0, 0, 0};
  int64_t prof_n[kPhases] = {0, 0, 0, 0, 0};
  bool phase_timing = false;
  int64_t cyc_cap = 0;            // rows per array of d_cyc
  double *d_cyc = nullptr;        // [2 x cyc_cap]: per-row Gram and solve cycles
  double *d_cyc_sum = nullptr;    // [2]
  double *h_cyc_sum = nullptr;    // pinned [2]
  double cyc[2][2] = {{0, 0}, {0, 0}};  // per side: Gram, solve
  int64_t n_hold = -1;             // held-out pairs (-1: none registered)
  int32_t *d_hu = nullptr;         // held-out users, items and ratings, in CSR order
  int32_t *d_hi = nullptr;
  uint8_t *d_hr = nullptr;
  double *d_hold_blocks = nullptr; // per-block squared errors
  double *d_hold_partials = nullptr;
  double *d_hold_sse = nullptr;
  // tensor ALS over time bins (als_set_time_bins)
  int32_t n_bins = 0;
  int32_t *d_tbin = nullptr;       // time bin of every rating, CSR order
  int32_t *d_tbin_t = nullptr;     // the same in CSC order
  std::vector<int64_t> h_tb_ptr;   // ratings grouped by time bin
  int64_t *d_tb_ptr = nullptr;
  int32_t *d_tb_user = nullptr, *d_tb_item = nullptr;
  uint8_t *d_tb_val = nullptr;
  float *d_fpad2 = nullptr;        // second staged table [(max(M, N, bins) + 1) x DP]
  // Bayesian Gibbs step (allocated on first use)
  float *d_prior_init = nullptr;   // prior image of the row kernels
  float *d_prior_K = nullptr;      // Cholesky factor of the prior precision (rows without ratings)
  float *d_prior_mu32 = nullptr;
  int32_t *d_prior_ok = nullptr;
  double *d_bayes_scratch = nullptr;
  double *d_hyper_partials = nullptr;
  int32_t *d_hyper_status = nullptr;
  int32_t *h_hyper_status = nullptr;  // pinned
  // Normal-Wishart hyperprior per side: users, items, and (BPTF) the time chain
  double *d_nw_mu0[3] = {nullptr, nullptr, nullptr};
  double *d_nw_W0inv[3] = {nullptr, nullptr, nullptr};
  double nw_beta0[3] = {0, 0, 0}, nw_nu0[3] = {0, 0, 0};
  bool nw_set[3] = {false, false, false};
  // BPTF time chain (allocated on first use)
  float *d_time_h0 = nullptr;      // per-bin prior right-hand side [n_bins x D]
  int64_t time_h0_bins = 0;
  double *d_time_extra = nullptr;  // step scatter of the chain, D (D + 1) / 2
  double *d_time_partials = nullptr;  // its per-slice partial sums
  int64_t time_partials_cap = 0;
  double *d_zero_mu = nullptr;     // D zeros (the chain's image has no mean term)
  double *d_scratch = nullptr;     // this device's copy of the allocation-free scratch array
};

namespace {

thread_local std::string g_create_err;

als_status fail(als_ctx *ctx, als_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (ctx) ctx->err = buf; else g_create_err = buf;
  return st;
}

#define HIP_OR_FAIL(ctx, call)                                                              \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return fail((ctx), e_ == hipErrorOutOfMemory ? ALS_ERR_OUT_OF_MEMORY : ALS_ERR_HIP,    \
                  "%s failed: %s", #call, hipGetErrorString(e_));                           \
  } while (0)

template <typename T>
hipError_t dalloc(T **p, int64_t n) {
  *p = nullptr;
  return hipMalloc((void **)p, sizeof(T) * (size_t)std::max<int64_t>(n, 1));
}

template <typename T>
void dfree(T *&p) {
  if (p) (void)hipFree((void *)p);
  p = nullptr;
}

struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) == hipSuccess && prev != dev) (void)hipSetDevice(dev);
  }
  ~DeviceGuard() {
    int cur;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

size_t slot_bytes_of(const als_ctx *ctx) {
  return ctx->lane_solve ? (size_t)als::ne_floats(als::lane_width(ctx->D)) * sizeof(float)
                         : als::slot_floats_rt(ctx->DP) * sizeof(float);
}

// Degree-ordered schedule of one side with hub rows split into chunks.
// Row blocking of the device transpose: blocks of rows_per_blk rows whose per-column
// counters (nblk x n_items int32) stay within kCscTableEntries.
void csc_blocking(int64_t n_users, int64_t n_items, int64_t &rows_per_blk, int64_t &nblk) {
  const int64_t max_blk = std::max<int64_t>(1, kCscTableEntries / std::max<int64_t>(n_items, 1));
  rows_per_blk = std::max<int64_t>(16, (n_users + max_blk - 1) / max_blk);
  nblk = (n_users + rows_per_blk - 1) / rows_per_blk;
}

// parity >= 0: only the rows s with s % 2 == parity, and those without ratings are
// scheduled like the others (the time chain's bins, whose prior depends on the row).
als_status build_plan(als_ctx *ctx, SidePlan &P, const std::vector<int64_t> &ptr,
                      int parity = -1) {
  const int64_t n_rows = (int64_t)ptr.size() - 1;
  P = SidePlan();
  P.n_rows = n_rows;
  std::vector<int32_t> order;
  order.reserve(n_rows);
  for (int64_t s = 0; s < n_rows; ++s) {
    const int64_t d = ptr[s + 1] - ptr[s];
    if (parity >= 0) {
      if ((s & 1) != parity) continue;
      order.push_back((int32_t)s);
    } else if (d > 0) {
      order.push_back((int32_t)s);
    } else {
      P.zero_rows.push_back((int32_t)s);
    }
    P.max_deg = std::max(P.max_deg, d);
  }
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    return ptr[a + 1] - ptr[a] > ptr[b + 1] - ptr[b];
  });
  P.rows_with = (int64_t)order.size();
  const int64_t hub = ctx->tune.hub_threshold, chunk = ctx->tune.chunk;
  const int64_t cap = std::max<int64_t>(1, ctx->tune.workspace_bytes / (int64_t)slot_bytes_of(ctx));
  const int64_t max_chunks = P.max_deg > hub ? (P.max_deg + chunk - 1) / chunk : 0;
  if (max_chunks > cap)
    return fail(ctx, ALS_ERR_INVALID_ARG,
                "workspace of %lld bytes holds %lld slots; a split row needs %lld",
                (long long)ctx->tune.workspace_bytes, (long long)cap, (long long)max_chunks);
  // batches of consecutive rows whose chunks fit the workspace
  std::vector<std::pair<int64_t, int64_t>> spans;  // [first, last) positions in order
  {
    int64_t first = 0, slots = 0;
    for (int64_t k = 0; k < (int64_t)order.size(); ++k) {
      const int64_t d = ptr[order[k] + 1] - ptr[order[k]];
      const int64_t nch = d > hub ? (d + chunk - 1) / chunk : 0;
      if (slots + nch > cap) {
        spans.push_back({first, k});
        first = k;
        slots = 0;
      }
      slots += nch;
    }
    if (first < (int64_t)order.size()) spans.push_back({first, (int64_t)order.size()});
  }
  for (const auto &sp : spans) {
    Batch b{(int64_t)P.gitems.size(), 0, 0, (int64_t)P.rows.size(), 0, 0, 0};
    // chunks of the batch's split rows
    for (int64_t k = sp.first; k < sp.second; ++k) {
      const int32_t s = order[k];
      const int64_t d = ptr[s + 1] - ptr[s];
      if (d <= hub) continue;
      const int64_t nch = (d + chunk - 1) / chunk;
      ++P.split_rows;
      RowTask rt;
      rt.start = ptr[s];
      rt.slot0 = b.n_slots;
      rt.row = s;
      rt.deg = (int32_t)d;
      rt.nslots = (int32_t)nch;
      rt.sse_idx = -1;
      P.rows.push_back(rt);
      for (int64_t q = 0; q < nch; ++q) {
        WorkItem it;
        it.start = ptr[s] + q * chunk;
        it.len = (int32_t)std::min<int64_t>(chunk, d - q * chunk);
        it.row = s;
        it.slot = b.n_slots + q;
        P.gitems.push_back(it);
      }
      b.n_slots += nch;
      b.n_gchunks += nch;
      b.n_split += 1;
    }
    // unsplit rows, one gather item each
    for (int64_t k = sp.first; k < sp.second; ++k) {
      const int32_t s = order[k];
      const int64_t d = ptr[s + 1] - ptr[s];
      if (d > hub) continue;
      RowTask rt;
      rt.start = ptr[s];
      rt.slot0 = (int64_t)P.rows.size();  // record of the row's packed normal equations
      rt.row = s;
      rt.deg = (int32_t)d;
      rt.nslots = 0;
      rt.sse_idx = (int32_t)P.gitems.size();
      P.rows.push_back(rt);
      WorkItem it;
      it.start = ptr[s];
      it.len = (int32_t)d;
      it.row = s;
      it.slot = rt.slot0;
      P.gitems.push_back(it);
    }
    b.n_gitems = (int64_t)P.gitems.size() - b.gitem_off;
    b.n_rows = (int64_t)P.rows.size() - b.row_off;
    P.n_chunks += b.n_gchunks;
    P.batches.push_back(b);
  }
  for (const Batch &b : P.batches) P.max_slots = std::max(P.max_slots, b.n_slots);
  HIP_OR_FAIL(ctx, dalloc(&P.d_gitems, (int64_t)P.gitems.size()));
  HIP_OR_FAIL(ctx, dalloc(&P.d_rows, (int64_t)P.rows.size()));
  HIP_OR_FAIL(ctx, dalloc(&P.d_zero_rows, (int64_t)P.zero_rows.size()));
  if (!P.zero_rows.empty())
    HIP_OR_FAIL(ctx, hipMemcpy(P.d_zero_rows, P.zero_rows.data(),
                               sizeof(int32_t) * P.zero_rows.size(), hipMemcpyHostToDevice));
  if (!P.gitems.empty())
    HIP_OR_FAIL(ctx, hipMemcpy(P.d_gitems, P.gitems.data(), sizeof(WorkItem) * P.gitems.size(),
                               hipMemcpyHostToDevice));
  if (!P.rows.empty())
    HIP_OR_FAIL(ctx, hipMemcpy(P.d_rows, P.rows.data(), sizeof(RowTask) * P.rows.size(),
                               hipMemcpyHostToDevice));
  return ALS_OK;
}

// pairs of one predict call: the launch has pair_blocks(n, D) < 2^31 blocks (with up to 8
// lanes per pair)
constexpr int64_t kMaxPairs = 0x7fffffffLL * 256 / 8;

void free_holdout(als_ctx *c) {
  dfree(c->d_hu);
  dfree(c->d_hi);
  dfree(c->d_hr);
  dfree(c->d_hold_blocks);
  dfree(c->d_hold_partials);
  dfree(c->d_hold_sse);
  c->n_hold = -1;
}

void free_ctx(als_ctx *c) {
  if (!c) return;
  DeviceGuard g(c->device);
  dfree(c->d_row_ptr);
  dfree(c->d_col);
  dfree(c->d_val);
  dfree(c->d_col_ptr);
  dfree(c->d_row_idx);
  dfree(c->d_val_t);
  dfree(c->d_w);
  dfree(c->d_w_t);
  for (auto &P : c->plan) {
    dfree(P.d_gitems);
    dfree(P.d_rows);
    dfree(P.d_zero_rows);
  }
  dfree(c->d_ws);
  dfree(c->d_fpad);
  dfree(c->d_ne);
  dfree(c->d_sse_items);
  dfree(c->d_partials);
  dfree(c->d_sse_in);
  dfree(c->d_sse_total);
  dfree(c->d_flag);
  if (c->h_sse) (void)hipHostFree(c->h_sse);
  if (c->h_sse_in) (void)hipHostFree(c->h_sse_in);
  if (c->h_flag) (void)hipHostFree(c->h_flag);
  dfree(c->d_cyc);
  dfree(c->d_cyc_sum);
  free_holdout(c);
  dfree(c->d_tbin);
  dfree(c->d_tbin_t);
  dfree(c->d_tb_ptr);
  dfree(c->d_tb_user);
  dfree(c->d_tb_item);
  dfree(c->d_tb_val);
  dfree(c->d_fpad2);
  dfree(c->d_prior_init);
  dfree(c->d_prior_K);
  dfree(c->d_prior_mu32);
  dfree(c->d_prior_ok);
  dfree(c->d_bayes_scratch);
  dfree(c->d_hyper_partials);
  dfree(c->d_hyper_status);
  if (c->h_hyper_status) (void)hipHostFree(c->h_hyper_status);
  for (int sd = 0; sd < 3; ++sd) {
    dfree(c->d_nw_mu0[sd]);
    dfree(c->d_nw_W0inv[sd]);
  }
  dfree(c->d_time_h0);
  dfree(c->d_time_extra);
  dfree(c->d_time_partials);
  dfree(c->d_zero_mu);
  if (c->h_cyc_sum) (void)hipHostFree(c->h_cyc_sum);
  for (auto &pe : c->prof_pending) {
    (void)hipEventDestroy(pe.a);
    (void)hipEventDestroy(pe.b);
  }
  for (auto e : c->ev_pool) (void)hipEventDestroy(e);
  delete c;
}

// ---- optional per-phase timing -------------------------------------------------------

hipEvent_t take_event(als_ctx *c) {
  if (!c->ev_pool.empty()) {
    hipEvent_t e = c->ev_pool.back();
    c->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

struct PhaseTimer {
  als_ctx *c;
  int phase;
  hipEvent_t a = nullptr;
  PhaseTimer(als_ctx *ctx, int ph) : c(ctx), phase(ph) {
    // mode 2 times only the gather kernels and, above D = 20, the fused row kernel
    const bool on = c->profiling && (c->prof_mode == 1 || ph == 1 || (ph == 2 && !c->lane_solve));
    if (on && (a = take_event(c))) (void)hipEventRecord(a, c->stream);
  }
  ~PhaseTimer() {
    if (!a) return;
    hipEvent_t b = take_event(c);
    if (!b) return;
    (void)hipEventRecord(b, c->stream);
    c->prof_pending.push_back(ProfEvent{phase, a, b});
  }
};

als_status collect_profile(als_ctx *c) {
  if (c->prof_pending.empty()) return ALS_OK;
  HIP_OR_FAIL(c, hipStreamSynchronize(c->stream));
  for (auto &pe : c->prof_pending) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, pe.a, pe.b) == hipSuccess) {
      c->prof_ms[pe.phase] += ms;
      c->prof_n[pe.phase] += 1;
    }
    c->ev_pool.push_back(pe.a);
    c->ev_pool.push_back(pe.b);
  }
  c->prof_pending.clear();
  return ALS_OK;
}

bool overlap(const void *a, size_t na, const void *b, size_t nb) {
  const char *pa = (const char *)a, *pb = (const char *)b;
  return pa < pb + nb && pb < pa + na;
}

// New-state residual pass over a side's pieces + fixed-order reduction into
// d_sse_total; the fixed side must already be staged in d_fpad.
// n_fixed: the rows of the staged fixed side (d_fpad), whose next row is the zero row.
als_status residual_pass(als_ctx *c, const SidePlan &P, const int32_t *idx, const uint8_t *val,
                         int64_t n_fixed, const float *X,
                         const als::Hadamard &hd = als::Hadamard{}) {
  const int64_t n = (int64_t)P.gitems.size();
  {
    PhaseTimer t(c, 3);
    HIP_OR_FAIL(c, als::launch_resid(c->DP, P.d_gitems, n, idx, val, c->d_fpad, n_fixed, X,
                                     c->D, c->d_sse_items, hd, c->stream));
  }
  {
    PhaseTimer t(c, 4);
    HIP_OR_FAIL(c, als::launch_reduce(c->d_sse_items, n, c->d_partials, c->d_sse_total,
                                      c->stream));
  }
  return ALS_OK;
}

// ---- scratch of the allocation-free validation RMSE ---------------------------------------
// als_pair_rmse_noalloc keeps the per-block squared errors of its pairs, the reduction's
// partial sums and the total in this file-scope array: every GPU the library runs on holds
// its own copy until the process ends. Host code never names the array itself (its name
// on the host is only a stand-in); it uses the device address that hipGetSymbolAddress
// returns for the current device, once per device, at context creation.
constexpr int64_t kScratchDoubles = 1 << 19;  // 4 MiB per GPU
constexpr int64_t kNoAllocMaxPairs = 16000000;
static __device__ __align__(256) double scratch[kScratchDoubles];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
double *g_scratch_dev[kMaxDevices] = {};

// Device address of the scratch array on `device`, which must be the current device.
hipError_t scratch_address(int device, double **out) {
  *out = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[device]) {
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_dev[device] = static_cast<double *>(ptr);
  }
  *out = g_scratch_dev[device];
  return hipSuccess;
}

}  // namespace

extern "C" {

const char *als_status_str(als_status s) {
  switch (s) {
    case ALS_OK: return "ok";
    case ALS_ERR_INVALID_ARG: return "invalid argument";
    case ALS_ERR_BAD_MATRIX: return "invalid rating matrix";
    case ALS_ERR_OUT_OF_MEMORY: return "out of memory";
    case ALS_ERR_HIP: return "HIP runtime error";
    case ALS_ERR_NOT_SPD: return "some rows were not positive definite and were left unchanged";
  }
  return "unknown status";
}

const char *als_last_error(const als_ctx *ctx) {
  return ctx ? ctx->err.c_str() : g_create_err.c_str();
}

als_status als_create(als_ctx **out, int64_t n_users, int64_t n_items, int64_t nnz,
                      const int64_t *row_ptr, const int32_t *col_idx, const uint8_t *ratings,
                      int32_t D, void *hip_stream, const als_tuning *tuning) {
  g_create_err.clear();
  if (!out) return fail(nullptr, ALS_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (n_users < 1 || n_items < 1 || n_users >= (1LL << 31) || n_items >= (1LL << 31))
    return fail(nullptr, ALS_ERR_INVALID_ARG, "matrix shape %lld x %lld out of range",
                (long long)n_users, (long long)n_items);
  if (nnz < 0 || nnz >= (1LL << 31))
    return fail(nullptr, ALS_ERR_INVALID_ARG, "nnz %lld out of range", (long long)nnz);
  if (D < 1 || D > 128) return fail(nullptr, ALS_ERR_INVALID_ARG, "D = %d outside [1, 128]", D);
  if ((std::max(n_users, n_items) + 1) * (int64_t)als::padded_width(D) * 4 > als::kMaxStagedBytes)
    return fail(nullptr, ALS_ERR_INVALID_ARG,
                "(max(n_users, n_items) + 1) * %d * 4 bytes exceeds the 4 GiB staged-factor limit",
                als::padded_width(D));
  if (!row_ptr || (nnz > 0 && (!col_idx || !ratings)))
    return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL host array");
  // ---- A1: validation of the CSR ----
  if (row_ptr[0] != 0) return fail(nullptr, ALS_ERR_BAD_MATRIX, "row_ptr[0] = %lld, expected 0",
                                   (long long)row_ptr[0]);
  if (row_ptr[n_users] != nnz)
    return fail(nullptr, ALS_ERR_BAD_MATRIX, "row_ptr[n_users] = %lld, expected nnz = %lld",
                (long long)row_ptr[n_users], (long long)nnz);
  for (int64_t u = 0; u < n_users; ++u) {
    if (row_ptr[u + 1] < row_ptr[u] || row_ptr[u + 1] > nnz)
      return fail(nullptr, ALS_ERR_BAD_MATRIX, "row_ptr decreases or exceeds nnz at row %lld",
                  (long long)u);
  }
  for (int64_t u = 0; u < n_users; ++u) {
    const int64_t a = row_ptr[u], b = row_ptr[u + 1];
    int64_t prev = -1;
    for (int64_t p = a; p < b; ++p) {
      const int64_t cidx = col_idx[p];
      if (cidx < 0 || cidx >= n_items)
        return fail(nullptr, ALS_ERR_BAD_MATRIX, "column %lld out of range at position %lld",
                    (long long)cidx, (long long)p);
      if (cidx <= prev)
        return fail(nullptr, ALS_ERR_BAD_MATRIX,
                    "columns not strictly increasing in row %lld (duplicate or unsorted)",
                    (long long)u);
      prev = cidx;
    }
  }
  als_ctx *c = new (std::nothrow) als_ctx();
  if (!c) return fail(nullptr, ALS_ERR_OUT_OF_MEMORY, "host allocation failed");
  c->M = n_users;
  c->N = n_items;
  c->nnz = nnz;
  c->D = D;
  c->DP = als::padded_width(D);
  c->lane_solve = als::lane_width(D) > 0;
  c->stream = (hipStream_t)hip_stream;
  c->tune.hub_threshold = kDefaultHubThreshold;
  c->tune.chunk = kDefaultChunk;
  c->tune.workspace_bytes = kDefaultWorkspace;
  if (tuning) {
    if (tuning->hub_threshold < 0 || tuning->chunk < 0 || tuning->workspace_bytes < 0) {
      delete c;
      return fail(nullptr, ALS_ERR_INVALID_ARG, "negative tuning value");
    }
    if (tuning->hub_threshold) c->tune.hub_threshold = tuning->hub_threshold;
    if (tuning->chunk) c->tune.chunk = tuning->chunk;
    if (tuning->workspace_bytes) c->tune.workspace_bytes = tuning->workspace_bytes;
  }
  if (hipGetDevice(&c->device) != hipSuccess) {
    delete c;
    return fail(nullptr, ALS_ERR_HIP, "no HIP device");
  }
  {
    const hipError_t e = scratch_address(c->device, &c->d_scratch);
    if (e != hipSuccess) {
      delete c;
      return fail(nullptr, ALS_ERR_HIP, "scratch address on device %d: %s", c->device,
                  hipGetErrorString(e));
    }
  }
  auto bail = [&](als_status st) {
    g_create_err = c->err;
    free_ctx(c);
    return st;
  };
#define CK(call)                                                                            \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess) {                                                                 \
      fail(c, e_ == hipErrorOutOfMemory ? ALS_ERR_OUT_OF_MEMORY : ALS_ERR_HIP,              \
           "%s failed: %s", #call, hipGetErrorString(e_));                                  \
      return bail(e_ == hipErrorOutOfMemory ? ALS_ERR_OUT_OF_MEMORY : ALS_ERR_HIP);         \
    }                                                                                       \
  } while (0)

  c->h_row_ptr.assign(row_ptr, row_ptr + n_users + 1);
  CK(dalloc(&c->d_row_ptr, n_users + 1));
  CK(dalloc(&c->d_col, nnz));
  CK(dalloc(&c->d_val, nnz));
  CK(dalloc(&c->d_col_ptr, n_items + 1));
  CK(dalloc(&c->d_row_idx, nnz));
  CK(dalloc(&c->d_val_t, nnz));
  CK(hipMemcpyAsync(c->d_row_ptr, row_ptr, sizeof(int64_t) * (n_users + 1),
                    hipMemcpyHostToDevice, c->stream));
  if (nnz > 0) {
    CK(hipMemcpyAsync(c->d_col, col_idx, sizeof(int32_t) * nnz, hipMemcpyHostToDevice,
                      c->stream));
    CK(hipMemcpyAsync(c->d_val, ratings, nnz, hipMemcpyHostToDevice, c->stream));
  }
  // ---- A2: device transpose ----
  {
    int64_t rows_per_blk = 0, nblk = 0;
    csc_blocking(n_users, n_items, rows_per_blk, nblk);
    int32_t *cnt = nullptr;
    int64_t *tot = nullptr;
    CK(dalloc(&cnt, nblk * n_items));
    CK(dalloc(&tot, n_items));
    hipError_t e = als::launch_csc_build(c->d_row_ptr, c->d_col, c->d_val, n_users, n_items,
                                         rows_per_blk, nblk, cnt, tot, c->d_col_ptr,
                                         c->d_row_idx, c->d_val_t, c->stream);
    hipError_t e2 = hipStreamSynchronize(c->stream);
    (void)hipFree(cnt);
    (void)hipFree(tot);
    CK(e);
    CK(e2);
  }
  c->h_col_ptr.resize(n_items + 1);
  CK(hipMemcpy(c->h_col_ptr.data(), c->d_col_ptr, sizeof(int64_t) * (n_items + 1),
               hipMemcpyDeviceToHost));
  if (c->h_col_ptr[n_items] != nnz) {
    fail(c, ALS_ERR_HIP, "device transpose produced %lld entries, expected %lld",
         (long long)c->h_col_ptr[n_items], (long long)nnz);
    return bail(ALS_ERR_HIP);
  }
  // ---- A3: schedules ----
  als_status st = build_plan(c, c->plan[ALS_ROWS_USERS], c->h_row_ptr);
  if (st != ALS_OK) return bail(st);
  st = build_plan(c, c->plan[ALS_ROWS_ITEMS], c->h_col_ptr);
  if (st != ALS_OK) return bail(st);
  int64_t max_slots = 0, max_sse = 0, max_rows = 0;
  for (auto &P : c->plan) {
    max_slots = std::max(max_slots, P.max_slots);
    max_sse = std::max(max_sse, (int64_t)P.gitems.size());
    max_rows = std::max(max_rows, (int64_t)P.rows.size());
  }
  c->ws_bytes = (size_t)max_slots * slot_bytes_of(c);
  CK(dalloc(&c->d_ws, (int64_t)(c->ws_bytes / sizeof(float))));
  if (c->lane_solve)
    CK(dalloc(&c->d_ne, max_rows * (int64_t)als::ne_floats(als::lane_width(D))));
  CK(dalloc(&c->d_fpad, (std::max(n_users, n_items) + 1) * (int64_t)c->DP));
  CK(dalloc(&c->d_sse_items, max_sse));
  CK(dalloc(&c->d_partials, als::reduce_partials(max_sse)));
  CK(dalloc(&c->d_sse_in, 1));
  CK(dalloc(&c->d_sse_total, 1));
  CK(dalloc(&c->d_flag, 1));
  CK(hipHostMalloc((void **)&c->h_sse, sizeof(double), hipHostMallocDefault));
  // written by the half-sweep's last reduction kernel, so coherent and mapped
  CK(hipHostMalloc((void **)&c->h_sse_in, 2 * sizeof(double),
                   hipHostMallocMapped | hipHostMallocCoherent));
  CK(hipHostMalloc((void **)&c->h_flag, sizeof(int32_t),
                   hipHostMallocMapped | hipHostMallocCoherent));
  CK(hipHostGetDevicePointer((void **)&c->hd_sse_in, c->h_sse_in, 0));
  CK(hipHostGetDevicePointer((void **)&c->hd_flag, c->h_flag, 0));
  *c->h_flag = 0;
  *c->h_sse = 0.0;
  c->h_sse_in[0] = c->h_sse_in[1] = 0.0;
  CK(als::launch_fill_i32(c->d_flag, 1, 0, c->stream));
  CK(hipStreamSynchronize(c->stream));
#undef CK
  *out = c;
  return ALS_OK;
}

}  // extern "C"

namespace {

// The half-sweep of both methods: the ALS update (pr.init == nullptr, lambda used) or the
// Gibbs draw (pr: the prior image, the variates and their scale; lambda unused).
// What a half-sweep reads: the plan (0 users, 1 items, 2 time bins), the side's index,
// rating and weight arrays, the rows of the staged table (its zero row) and, for tensor
// ALS, the second index and staged table.
struct SweepSpec {
  int plan = 0;
  const int32_t *idx = nullptr;
  const uint8_t *val = nullptr;
  const float *wts = nullptr;
  int64_t n_fixed = 0;
  als::Hadamard hd;
  bool keep_flags = false;  // add to the flag count of the previous sweep (time chain)
  int sse_in_part = 0;      // which part of the entering-state SSE this pass writes
};

als_status run_sweep(als_ctx *ctx, const SweepSpec &sp, float lambda, float *out_factors,
                     double *rmse_out, const als::RowPrior &pr);

als_status half_sweep_impl(als_ctx *ctx, als_side side, const float *fixed_factors, float lambda,
                           float *out_factors, double *rmse_out, const als::RowPrior &pr) {
  if (side != ALS_ROWS_USERS && side != ALS_ROWS_ITEMS)
    return fail(ctx, ALS_ERR_INVALID_ARG, "side %d is not ALS_ROWS_USERS or ALS_ROWS_ITEMS",
                (int)side);
  if (!fixed_factors || !out_factors) return fail(ctx, ALS_ERR_INVALID_ARG, "NULL factor buffer");
  if (!std::isfinite(lambda) || lambda < 0.f)
    return fail(ctx, ALS_ERR_INVALID_ARG, "lambda must be finite and >= 0");
  if (((uintptr_t)fixed_factors & 15) || ((uintptr_t)out_factors & 15))
    return fail(ctx, ALS_ERR_INVALID_ARG, "factor buffers must be 16-byte aligned");
  const bool users = side == ALS_ROWS_USERS;
  const int64_t n_rows = users ? ctx->M : ctx->N, n_fixed = users ? ctx->N : ctx->M;
  if (overlap(fixed_factors, sizeof(float) * n_fixed * ctx->D, out_factors,
              sizeof(float) * n_rows * ctx->D))
    return fail(ctx, ALS_ERR_INVALID_ARG, "out_factors overlaps fixed_factors");
  DeviceGuard g(ctx->device);
  SweepSpec sp;
  sp.plan = side;
  sp.idx = users ? ctx->d_col : ctx->d_row_idx;
  sp.val = users ? ctx->d_val : ctx->d_val_t;
  sp.wts = users ? ctx->d_w : ctx->d_w_t;
  sp.n_fixed = n_fixed;
  {
    PhaseTimer t(ctx, 0);
    HIP_OR_FAIL(ctx, als::launch_stage_fixed(fixed_factors, n_fixed, ctx->D, ctx->DP,
                                             ctx->d_fpad, ctx->stream));
  }
  return run_sweep(ctx, sp, lambda, out_factors, rmse_out, pr);
}

// The batches of one half-sweep on an already staged fixed side (d_fpad, and d_fpad2 for
// tensor ALS), the entering-state reduction, the flag count and, on request, the
// new-state RMSE.
als_status run_sweep(als_ctx *ctx, const SweepSpec &sp, float lambda, float *out_factors,
                     double *rmse_out, const als::RowPrior &pr) {
  const SidePlan &P = ctx->plan[sp.plan];
  const int32_t *idx = sp.idx;
  const uint8_t *val = sp.val;
  const float *wts = sp.wts;
  const int64_t n_fixed = sp.n_fixed;
  const als::Hadamard &hd = sp.hd;
  const int side = sp.plan;
  if (!sp.keep_flags) HIP_OR_FAIL(ctx, als::launch_fill_i32(ctx->d_flag, 1, 0, ctx->stream));
  for (const Batch &b : P.batches) {
    double *sse = ctx->d_sse_items + b.gitem_off;
    if (ctx->lane_solve) {
      {
        PhaseTimer t(ctx, 1);
        HIP_OR_FAIL(ctx, als::launch_gram_ne(ctx->D, P.d_gitems + b.gitem_off, b.n_gitems,
                                             b.n_gchunks, idx, val, wts, ctx->d_fpad, n_fixed,
                                             out_factors, ctx->d_ws, ctx->d_ne, sse, hd,
                                             ctx->stream));
      }
      {
        PhaseTimer t(ctx, 2);
        HIP_OR_FAIL(ctx, als::launch_solve_lane(ctx->D, P.d_rows + b.row_off, b.n_rows, b.n_split,
                                                b.row_off, ctx->d_ws, ctx->d_ne, lambda,
                                                out_factors, ctx->d_flag, pr, ctx->stream));
      }
    } else {
      if (b.n_gchunks > 0) {
        PhaseTimer t(ctx, 1);
        HIP_OR_FAIL(ctx, als::launch_gram_chunks(ctx->DP, P.d_gitems + b.gitem_off, b.n_gchunks,
                                                 idx, val, wts, ctx->d_fpad, n_fixed, out_factors,
                                                 ctx->D, ctx->d_ws, sse, hd, ctx->stream));
      }
      {
        PhaseTimer t(ctx, 2);
        const bool clocks = ctx->phase_timing && side < 2;  // the clocks cover users and items
        double *cg = clocks ? ctx->d_cyc + b.row_off : nullptr;
        double *cs = clocks ? ctx->d_cyc + ctx->cyc_cap + b.row_off : nullptr;
        HIP_OR_FAIL(ctx, als::launch_rows(ctx->DP, P.d_rows + b.row_off, b.n_rows, idx, val, wts,
                                          ctx->d_fpad, n_fixed, ctx->d_ws, ctx->D, lambda,
                                          out_factors, ctx->d_sse_items, ctx->d_flag, cg, cs,
                                          pr, hd, ctx->stream));
      }
    }
  }
  if (pr.init && !P.zero_rows.empty()) {
    PhaseTimer t(ctx, 2);
    HIP_OR_FAIL(ctx, als::launch_prior_rows(P.d_zero_rows, (int64_t)P.zero_rows.size(), ctx->D,
                                            ctx->d_prior_K, ctx->d_prior_mu32, ctx->d_prior_ok,
                                            pr.z, out_factors, ctx->d_flag, ctx->stream));
  }
  {
    PhaseTimer t(ctx, 4);
    HIP_OR_FAIL(ctx, als::launch_reduce(ctx->d_sse_items, (int64_t)P.gitems.size(),
                                        ctx->d_partials, ctx->d_sse_in, ctx->stream,
                                        ctx->hd_sse_in + sp.sse_in_part, ctx->d_flag,
                                        ctx->hd_flag));
  }
  ctx->last_side = side;
  ctx->sse_in_parts = sp.sse_in_part + 1;
  if (ctx->phase_timing && !ctx->lane_solve && !P.rows.empty() && side < 2) {
    const int64_t nr = (int64_t)P.rows.size();
    HIP_OR_FAIL(ctx, als::launch_reduce(ctx->d_cyc, nr, ctx->d_partials, ctx->d_cyc_sum,
                                        ctx->stream));
    HIP_OR_FAIL(ctx, als::launch_reduce(ctx->d_cyc + ctx->cyc_cap, nr, ctx->d_partials,
                                        ctx->d_cyc_sum + 1, ctx->stream));
    HIP_OR_FAIL(ctx, hipMemcpyAsync(ctx->h_cyc_sum, ctx->d_cyc_sum, 2 * sizeof(double),
                                    hipMemcpyDeviceToHost, ctx->stream));
    HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
    ctx->cyc[side][0] += ctx->h_cyc_sum[0];
    ctx->cyc[side][1] += ctx->h_cyc_sum[1];
  }
  if (rmse_out) {
    als_status st = residual_pass(ctx, P, idx, val, n_fixed, out_factors, hd);
    if (st != ALS_OK) return st;
    HIP_OR_FAIL(ctx, hipMemcpyAsync(ctx->h_sse, ctx->d_sse_total, sizeof(double),
                                    hipMemcpyDeviceToHost, ctx->stream));
    HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
    *rmse_out = ctx->nnz > 0 ? std::sqrt(*ctx->h_sse / (double)ctx->nnz) : 0.0;
    if (*ctx->h_flag > 0)
      return fail(ctx, ALS_ERR_NOT_SPD, "%d rows were flagged and left unchanged",
                  (int)*ctx->h_flag);
  }
  return ALS_OK;
}

template <typename T>
als_status ensure(als_ctx *ctx, T **p, size_t n, const char *what) {
  if (*p) return ALS_OK;
  const hipError_t e = dalloc(p, (int64_t)n);
  if (e != hipSuccess)
    return fail(ctx, e == hipErrorOutOfMemory ? ALS_ERR_OUT_OF_MEMORY : ALS_ERR_HIP, "%s: %s",
                what, hipGetErrorString(e));
  return ALS_OK;
}

als_status ensure_bayes(als_ctx *ctx) {
  const int D = ctx->D;
  als_status st = ensure(ctx, &ctx->d_prior_init, als::prior_init_floats(D, ctx->DP), "prior image");
  if (st == ALS_OK) st = ensure(ctx, &ctx->d_prior_K, (size_t)D * D, "prior factor");
  if (st == ALS_OK) st = ensure(ctx, &ctx->d_prior_mu32, (size_t)D, "prior mean");
  if (st == ALS_OK) st = ensure(ctx, &ctx->d_prior_ok, 1, "prior status");
  if (st == ALS_OK) st = ensure(ctx, &ctx->d_bayes_scratch, als::bayes_scratch_doubles(D), "scratch");
  if (st == ALS_OK)
    st = ensure(ctx, &ctx->d_hyper_partials,
                (size_t)als::hyper_blocks(std::max(ctx->M, ctx->N)) * als::hyper_entries(D),
                "moment partials");
  if (st == ALS_OK) st = ensure(ctx, &ctx->d_hyper_status, 1, "draw status");
  if (st == ALS_OK && !ctx->h_hyper_status) {
    const hipError_t e = hipHostMalloc((void **)&ctx->h_hyper_status, sizeof(int32_t),
                                       hipHostMallocDefault);
    if (e != hipSuccess) return fail(ctx, ALS_ERR_OUT_OF_MEMORY, "pinned status: %s",
                                     hipGetErrorString(e));
  }
  return st;
}

// The Normal-Wishart hyperprior of users (0), items (1) or the time chain (2).
als_status set_nw_prior_at(als_ctx *ctx, int at, const double *mu0, double beta0,
                           const double *W0_inv, double nu0) {
  const int D = ctx->D;
  if (!mu0 || !W0_inv) return fail(ctx, ALS_ERR_INVALID_ARG, "NULL argument");
  if (!(beta0 >= 0.0) || !std::isfinite(beta0) || !std::isfinite(nu0) || !(nu0 > D - 1))
    return fail(ctx, ALS_ERR_INVALID_ARG, "need beta0 >= 0 and nu0 > D - 1");
  for (int a = 0; a < D; ++a) {
    if (!std::isfinite(mu0[a])) return fail(ctx, ALS_ERR_INVALID_ARG, "mu0 is not finite");
    for (int e = 0; e < D; ++e) {
      if (!std::isfinite(W0_inv[a * D + e]) || W0_inv[a * D + e] != W0_inv[e * D + a])
        return fail(ctx, ALS_ERR_INVALID_ARG, "W0_inv must be finite and symmetric");
    }
  }
  DeviceGuard g(ctx->device);
  als_status st = ensure(ctx, &ctx->d_nw_mu0[at], (size_t)D, "prior mean");
  if (st == ALS_OK) st = ensure(ctx, &ctx->d_nw_W0inv[at], (size_t)D * D, "prior scale");
  if (st != ALS_OK) return st;
  HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
  HIP_OR_FAIL(ctx, hipMemcpy(ctx->d_nw_mu0[at], mu0, sizeof(double) * D, hipMemcpyHostToDevice));
  HIP_OR_FAIL(ctx, hipMemcpy(ctx->d_nw_W0inv[at], W0_inv, sizeof(double) * D * D,
                             hipMemcpyHostToDevice));
  ctx->nw_beta0[at] = beta0;
  ctx->nw_nu0[at] = nu0;
  ctx->nw_set[at] = true;
  return ALS_OK;
}

}  // namespace

extern "C" {

als_status als_half_sweep(als_ctx *ctx, als_side side, const float *fixed_factors, float lambda,
                          float *out_factors, double *rmse_out) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  return half_sweep_impl(ctx, side, fixed_factors, lambda, out_factors, rmse_out, als::RowPrior{});
}

als_status als_gibbs_half_sweep(als_ctx *ctx, als_side side, const float *fixed_factors,
                                float alpha, const double *Lambda, const double *mu,
                                const float *z, float *out_factors, double *rmse_out) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (!(alpha > 0.f) || !std::isfinite(alpha))
    return fail(ctx, ALS_ERR_INVALID_ARG, "alpha must be finite and > 0");
  if (!Lambda || !mu || !z) return fail(ctx, ALS_ERR_INVALID_ARG, "NULL prior or variates");
  if (side != ALS_ROWS_USERS && side != ALS_ROWS_ITEMS)
    return fail(ctx, ALS_ERR_INVALID_ARG, "side %d is not ALS_ROWS_USERS or ALS_ROWS_ITEMS",
                (int)side);
  if ((side == ALS_ROWS_USERS ? ctx->d_w : ctx->d_w_t) != nullptr)
    return fail(ctx, ALS_ERR_INVALID_ARG, "the Gibbs half-sweep takes no rating weights; detach them");
  const int64_t n_rows = side == ALS_ROWS_USERS ? ctx->M : ctx->N;
  if (overlap(z, sizeof(float) * n_rows * ctx->D, out_factors, sizeof(float) * n_rows * ctx->D))
    return fail(ctx, ALS_ERR_INVALID_ARG, "z overlaps out_factors");
  DeviceGuard g(ctx->device);
  als_status st = ensure_bayes(ctx);
  if (st != ALS_OK) return st;
  HIP_OR_FAIL(ctx, als::launch_prior_prepare(Lambda, mu, ctx->D, ctx->DP, (double)alpha,
                                             !ctx->plan[side].zero_rows.empty(),
                                             ctx->d_prior_init, ctx->d_prior_K, ctx->d_prior_mu32,
                                             ctx->d_prior_ok, ctx->stream));
  als::RowPrior pr;
  pr.init = ctx->d_prior_init;
  pr.z = z;
  pr.zscale = (float)(1.0 / std::sqrt((double)alpha));
  return half_sweep_impl(ctx, side, fixed_factors, 0.f, out_factors, rmse_out, pr);
}

als_status als_set_nw_prior(als_ctx *ctx, als_side side, const double *mu0, double beta0,
                            const double *W0_inv, double nu0) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (side != ALS_ROWS_USERS && side != ALS_ROWS_ITEMS)
    return fail(ctx, ALS_ERR_INVALID_ARG, "side must be ALS_ROWS_USERS or ALS_ROWS_ITEMS");
  return set_nw_prior_at(ctx, (int)side, mu0, beta0, W0_inv, nu0);
}

als_status als_set_time_nw_prior(als_ctx *ctx, const double *mu0, double beta0,
                                 const double *W0_inv, double nu0) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  return set_nw_prior_at(ctx, 2, mu0, beta0, W0_inv, nu0);
}

als_status als_sample_hyper(als_ctx *ctx, als_side side, const float *X, const double *chi2,
                            const double *offdiag, const double *z_mu, double *mu_out,
                            double *Lambda_out, int32_t *status_out) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (side != ALS_ROWS_USERS && side != ALS_ROWS_ITEMS)
    return fail(ctx, ALS_ERR_INVALID_ARG, "side must be ALS_ROWS_USERS or ALS_ROWS_ITEMS");
  if (!ctx->nw_set[side]) return fail(ctx, ALS_ERR_INVALID_ARG, "no Normal-Wishart prior set for this side");
  if (!X || !chi2 || (!offdiag && ctx->D > 1) || !z_mu || !mu_out || !Lambda_out)
    return fail(ctx, ALS_ERR_INVALID_ARG, "NULL argument");
  if ((uintptr_t)X & 15) return fail(ctx, ALS_ERR_INVALID_ARG, "X must be 16-byte aligned");
  const int64_t n = side == ALS_ROWS_USERS ? ctx->M : ctx->N;
  DeviceGuard g(ctx->device);
  als_status st = ensure_bayes(ctx);
  if (st != ALS_OK) return st;
  const int nblk = als::hyper_blocks(n);
  HIP_OR_FAIL(ctx, als::launch_hyper_moments(X, n, ctx->D, ctx->d_hyper_partials, ctx->stream));
  HIP_OR_FAIL(ctx, als::launch_hyper_sample(ctx->d_hyper_partials, nblk, n, ctx->D,
                                            ctx->d_nw_mu0[side], ctx->nw_beta0[side],
                                            ctx->d_nw_W0inv[side], ctx->nw_nu0[side], chi2,
                                            offdiag, z_mu, ctx->d_bayes_scratch, mu_out,
                                            Lambda_out, ctx->d_hyper_status, ctx->stream));
  if (status_out) {
    HIP_OR_FAIL(ctx, hipMemcpyAsync(ctx->h_hyper_status, ctx->d_hyper_status, sizeof(int32_t),
                                    hipMemcpyDeviceToHost, ctx->stream));
    HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
    *status_out = *ctx->h_hyper_status;
    if (*status_out != 0)
      return fail(ctx, ALS_ERR_NOT_SPD, "a factorisation of the Normal-Wishart draw failed");
  }
  return ALS_OK;
}

als_status als_last_rmse_in(als_ctx *ctx, double *rmse_in) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (!rmse_in) return fail(ctx, ALS_ERR_INVALID_ARG, "NULL argument");
  if (ctx->last_side < 0) return fail(ctx, ALS_ERR_INVALID_ARG, "no half-sweep has run yet");
  DeviceGuard g(ctx->device);
  HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
  // the time chain's passes cover disjoint ratings (a rating's prediction reads only its own
  // bin's row, which the other parity's pass leaves alone): their parts add up, in order
  double sse = 0.0;
  for (int q = 0; q < ctx->sse_in_parts; ++q) sse += ctx->h_sse_in[q];
  *rmse_in = ctx->nnz > 0 ? std::sqrt(sse / (double)ctx->nnz) : 0.0;
  return ALS_OK;
}

als_status als_rmse(als_ctx *ctx, const float *U, const float *V, double *rmse_out) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (!U || !V || !rmse_out) return fail(ctx, ALS_ERR_INVALID_ARG, "NULL argument");
  if (((uintptr_t)U & 15) || ((uintptr_t)V & 15))
    return fail(ctx, ALS_ERR_INVALID_ARG, "factor buffers must be 16-byte aligned");
  DeviceGuard g(ctx->device);
  const SidePlan &P = ctx->plan[ALS_ROWS_USERS];
  {
    PhaseTimer t(ctx, 0);
    HIP_OR_FAIL(ctx, als::launch_stage_fixed(V, ctx->N, ctx->D, ctx->DP, ctx->d_fpad,
                                             ctx->stream));
  }
  als_status st = residual_pass(ctx, P, ctx->d_col, ctx->d_val, ctx->N, U);
  if (st != ALS_OK) return st;
  HIP_OR_FAIL(ctx, hipMemcpyAsync(ctx->h_sse, ctx->d_sse_total, sizeof(double),
                                  hipMemcpyDeviceToHost, ctx->stream));
  HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
  *rmse_out = ctx->nnz > 0 ? std::sqrt(*ctx->h_sse / (double)ctx->nnz) : 0.0;
  return ALS_OK;
}

int64_t als_flagged_rows(const als_ctx *ctx) {
  if (!ctx) return -1;
  DeviceGuard g(ctx->device);
  if (hipStreamSynchronize(ctx->stream) != hipSuccess) return -1;
  return *ctx->h_flag;
}

als_status als_get_csc(als_ctx *ctx, int64_t *col_ptr, int32_t *row_idx, uint8_t *ratings) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (!col_ptr || (ctx->nnz > 0 && (!row_idx || !ratings)))
    return fail(ctx, ALS_ERR_INVALID_ARG, "NULL host buffer");
  DeviceGuard g(ctx->device);
  HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
  HIP_OR_FAIL(ctx, hipMemcpy(col_ptr, ctx->d_col_ptr, sizeof(int64_t) * (ctx->N + 1),
                             hipMemcpyDeviceToHost));
  if (ctx->nnz > 0) {
    HIP_OR_FAIL(ctx, hipMemcpy(row_idx, ctx->d_row_idx, sizeof(int32_t) * ctx->nnz,
                               hipMemcpyDeviceToHost));
    HIP_OR_FAIL(ctx, hipMemcpy(ratings, ctx->d_val_t, ctx->nnz, hipMemcpyDeviceToHost));
  }
  return ALS_OK;
}

als_status als_plan_stats(als_ctx *ctx, als_side side, int64_t *out, int32_t n) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  if ((side != ALS_ROWS_USERS && side != ALS_ROWS_ITEMS) || !out || n < 0)
    return fail(ctx, ALS_ERR_INVALID_ARG, "bad argument");
  const SidePlan &P = ctx->plan[side];
  const int64_t v[7] = {P.rows_with, P.split_rows, P.n_chunks, (int64_t)P.batches.size(),
                        P.max_deg, (int64_t)ctx->ws_bytes, (int64_t)slot_bytes_of(ctx)};
  for (int32_t i = 0; i < n && i < 7; ++i) out[i] = v[i];
  return ALS_OK;
}

als_status als_set_weights(als_ctx *ctx, const float *weights) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  DeviceGuard g(ctx->device);
  if (!weights) {
    HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
    dfree(ctx->d_w);
    dfree(ctx->d_w_t);
    return ALS_OK;
  }
  for (int64_t p = 0; p < ctx->nnz; ++p) {
    if (!(weights[p] >= 0.f) || !std::isfinite(weights[p]))
      return fail(ctx, ALS_ERR_INVALID_ARG, "weight %lld is not a finite non-negative number",
                  (long long)p);
  }
  const int64_t nnz = ctx->nnz;
  if (!ctx->d_w) {
    float *w = nullptr, *wt = nullptr;
    hipError_t e = dalloc(&w, nnz);
    if (e == hipSuccess) e = dalloc(&wt, nnz);
    if (e != hipSuccess) {
      dfree(w);
      dfree(wt);
      return fail(ctx, e == hipErrorOutOfMemory ? ALS_ERR_OUT_OF_MEMORY : ALS_ERR_HIP,
                  "weight buffers: %s", hipGetErrorString(e));
    }
    ctx->d_w = w;
    ctx->d_w_t = wt;
  }
  if (nnz == 0) return ALS_OK;
  HIP_OR_FAIL(ctx, hipMemcpyAsync(ctx->d_w, weights, sizeof(float) * nnz, hipMemcpyHostToDevice,
                                  ctx->stream));
  int64_t rows_per_blk = 0, nblk = 0;
  csc_blocking(ctx->M, ctx->N, rows_per_blk, nblk);
  int32_t *cnt = nullptr;
  int64_t *tot = nullptr;
  hipError_t e = dalloc(&cnt, nblk * ctx->N);
  if (e == hipSuccess) e = dalloc(&tot, ctx->N);
  if (e == hipSuccess)
    e = als::launch_csc_permute_f32(ctx->d_row_ptr, ctx->d_col, ctx->d_w, ctx->M, ctx->N,
                                    rows_per_blk, nblk, cnt, tot, ctx->d_col_ptr, ctx->d_w_t,
                                    ctx->stream);
  const hipError_t e2 = hipStreamSynchronize(ctx->stream);
  dfree(cnt);
  dfree(tot);
  HIP_OR_FAIL(ctx, e);
  HIP_OR_FAIL(ctx, e2);
  return ALS_OK;
}

als_status als_set_phase_timing(als_ctx *ctx, int32_t enable) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  DeviceGuard g(ctx->device);
  if (enable && !ctx->d_cyc) {
    const int64_t cap = std::max<int64_t>(
        1, std::max((int64_t)ctx->plan[0].rows.size(), (int64_t)ctx->plan[1].rows.size()));
    double *cyc = nullptr, *sum = nullptr, *host = nullptr;
    hipError_t e = dalloc(&cyc, 2 * cap);
    if (e == hipSuccess) e = dalloc(&sum, 2);
    if (e == hipSuccess) e = hipHostMalloc((void **)&host, 2 * sizeof(double), hipHostMallocDefault);
    if (e != hipSuccess) {
      dfree(cyc);
      dfree(sum);
      return fail(ctx, e == hipErrorOutOfMemory ? ALS_ERR_OUT_OF_MEMORY : ALS_ERR_HIP,
                  "phase timing buffers: %s", hipGetErrorString(e));
    }
    ctx->d_cyc = cyc;
    ctx->d_cyc_sum = sum;
    ctx->h_cyc_sum = host;
    ctx->cyc_cap = cap;
  }
  ctx->phase_timing = enable != 0;
  for (auto &side : ctx->cyc) side[0] = side[1] = 0.0;
  return ALS_OK;
}

als_status als_get_phase_cycles(als_ctx *ctx, als_side side, double *gram_cycles,
                                double *solve_cycles) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (side != ALS_ROWS_USERS && side != ALS_ROWS_ITEMS)
    return fail(ctx, ALS_ERR_INVALID_ARG, "side must be ALS_ROWS_USERS or ALS_ROWS_ITEMS");
  if (!gram_cycles || !solve_cycles) return fail(ctx, ALS_ERR_INVALID_ARG, "NULL argument");
  *gram_cycles = ctx->cyc[side][0];
  *solve_cycles = ctx->cyc[side][1];
  return ALS_OK;
}

// ---- tensor ALS over time bins ----------------------------------------------------------

als_status als_set_time_bins(als_ctx *ctx, int32_t n_bins, const int32_t *bins) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (n_bins < 1) return fail(ctx, ALS_ERR_INVALID_ARG, "n_bins must be >= 1");
  if (((int64_t)n_bins + 1) * ctx->DP * 4 > als::kMaxStagedBytes)
    return fail(ctx, ALS_ERR_INVALID_ARG, "too many time bins for the staged-table limit");
  if (ctx->nnz > 0 && !bins) return fail(ctx, ALS_ERR_INVALID_ARG, "NULL bins");
  for (int64_t p = 0; p < ctx->nnz; ++p) {
    if (bins[p] < 0 || bins[p] >= n_bins)
      return fail(ctx, ALS_ERR_INVALID_ARG, "time bin %d of rating %lld outside [0, %d)",
                  bins[p], (long long)p, n_bins);
  }
  DeviceGuard g(ctx->device);
  HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
  dfree(ctx->d_tbin);
  dfree(ctx->d_tbin_t);
  dfree(ctx->d_tb_ptr);
  dfree(ctx->d_tb_user);
  dfree(ctx->d_tb_item);
  dfree(ctx->d_tb_val);
  dfree(ctx->d_fpad2);
  for (int q = 2; q < 5; ++q) {
    SidePlan &P = ctx->plan[q];
    dfree(P.d_gitems);
    dfree(P.d_rows);
    dfree(P.d_zero_rows);
    P = SidePlan();
  }
  SidePlan &TP = ctx->plan[2];
  dfree(ctx->d_time_h0);
  ctx->time_h0_bins = 0;
  ctx->n_bins = 0;
  const int64_t nnz = ctx->nnz, M = ctx->M;
  HIP_OR_FAIL(ctx, dalloc(&ctx->d_tbin, nnz));
  HIP_OR_FAIL(ctx, dalloc(&ctx->d_tbin_t, nnz));
  HIP_OR_FAIL(ctx, dalloc(&ctx->d_tb_ptr, (int64_t)n_bins + 1));
  HIP_OR_FAIL(ctx, dalloc(&ctx->d_tb_user, nnz));
  HIP_OR_FAIL(ctx, dalloc(&ctx->d_tb_item, nnz));
  HIP_OR_FAIL(ctx, dalloc(&ctx->d_tb_val, nnz));
  HIP_OR_FAIL(ctx, dalloc(&ctx->d_fpad2,
                          (std::max({ctx->M, ctx->N, (int64_t)n_bins}) + 1) * (int64_t)ctx->DP));
  // ratings grouped by time bin: a stable counting sort on the host (users ascending, then
  // the CSR order within a user), so the layout is the same on every run
  std::vector<int32_t> col(nnz);
  std::vector<uint8_t> val(nnz);
  if (nnz > 0) {
    HIP_OR_FAIL(ctx, hipMemcpy(ctx->d_tbin, bins, sizeof(int32_t) * nnz, hipMemcpyHostToDevice));
    HIP_OR_FAIL(ctx, hipMemcpy(col.data(), ctx->d_col, sizeof(int32_t) * nnz,
                               hipMemcpyDeviceToHost));
    HIP_OR_FAIL(ctx, hipMemcpy(val.data(), ctx->d_val, nnz, hipMemcpyDeviceToHost));
  }
  std::vector<int64_t> &ptr = ctx->h_tb_ptr;
  ptr.assign((size_t)n_bins + 1, 0);
  for (int64_t p = 0; p < nnz; ++p) ptr[bins[p] + 1] += 1;
  for (int32_t t = 0; t < n_bins; ++t) ptr[t + 1] += ptr[t];
  {
    std::vector<int64_t> next(ptr.begin(), ptr.end() - 1);
    std::vector<int32_t> tu(nnz), ti(nnz);
    std::vector<uint8_t> tv(nnz);
    for (int64_t u = 0; u < M; ++u) {
      for (int64_t p = ctx->h_row_ptr[u]; p < ctx->h_row_ptr[u + 1]; ++p) {
        const int64_t q = next[bins[p]]++;
        tu[q] = (int32_t)u;
        ti[q] = col[p];
        tv[q] = val[p];
      }
    }
    HIP_OR_FAIL(ctx, hipMemcpy(ctx->d_tb_ptr, ptr.data(), sizeof(int64_t) * ptr.size(),
                               hipMemcpyHostToDevice));
    if (nnz > 0) {
      HIP_OR_FAIL(ctx, hipMemcpy(ctx->d_tb_user, tu.data(), sizeof(int32_t) * nnz,
                                 hipMemcpyHostToDevice));
      HIP_OR_FAIL(ctx, hipMemcpy(ctx->d_tb_item, ti.data(), sizeof(int32_t) * nnz,
                                 hipMemcpyHostToDevice));
      HIP_OR_FAIL(ctx, hipMemcpy(ctx->d_tb_val, tv.data(), nnz, hipMemcpyHostToDevice));
    }
  }
  // the bins in CSC (item) order, through the transpose's own permutation (columns are
  // distinct within a row, so the positions are those of the CSC build)
  if (nnz > 0) {
    int64_t rows_per_blk = 0, nblk = 0;
    csc_blocking(ctx->M, ctx->N, rows_per_blk, nblk);
    int32_t *cnt = nullptr;
    int64_t *tot = nullptr;
    hipError_t e = dalloc(&cnt, nblk * ctx->N);
    if (e == hipSuccess) e = dalloc(&tot, ctx->N);
    if (e == hipSuccess)
      e = als::launch_csc_permute_f32(ctx->d_row_ptr, ctx->d_col,
                                      reinterpret_cast<const float *>(ctx->d_tbin), ctx->M,
                                      ctx->N, rows_per_blk, nblk, cnt, tot, ctx->d_col_ptr,
                                      reinterpret_cast<float *>(ctx->d_tbin_t), ctx->stream);
    const hipError_t e2 = hipStreamSynchronize(ctx->stream);
    dfree(cnt);
    dfree(tot);
    HIP_OR_FAIL(ctx, e);
    HIP_OR_FAIL(ctx, e2);
  }
  als_status st = build_plan(ctx, TP, ptr);
  if (st == ALS_OK) st = build_plan(ctx, ctx->plan[3], ptr, 0);
  if (st == ALS_OK) st = build_plan(ctx, ctx->plan[4], ptr, 1);
  if (st != ALS_OK) return st;
  // shared buffers sized for the time-bin plans too
  int64_t max_slots = 0, max_sse = 0, max_rows = 0;
  for (auto &P : ctx->plan) {
    max_slots = std::max(max_slots, P.max_slots);
    max_sse = std::max(max_sse, (int64_t)P.gitems.size());
    max_rows = std::max(max_rows, (int64_t)P.rows.size());
  }
  if ((size_t)max_slots * slot_bytes_of(ctx) > ctx->ws_bytes) {
    dfree(ctx->d_ws);
    ctx->ws_bytes = (size_t)max_slots * slot_bytes_of(ctx);
    HIP_OR_FAIL(ctx, dalloc(&ctx->d_ws, (int64_t)(ctx->ws_bytes / sizeof(float))));
  }
  if (ctx->lane_solve && (int64_t)TP.rows.size() > 0) {
    // records: one per row of the largest plan (already sized at create for users/items)
    const int64_t have = std::max((int64_t)ctx->plan[0].rows.size(),
                                  (int64_t)ctx->plan[1].rows.size());
    if (max_rows > have) {
      dfree(ctx->d_ne);
      HIP_OR_FAIL(ctx, dalloc(&ctx->d_ne, max_rows * (int64_t)als::ne_floats(als::lane_width(ctx->D))));
    }
  }
  const int64_t had_sse = std::max((int64_t)ctx->plan[0].gitems.size(),
                                   (int64_t)ctx->plan[1].gitems.size());
  if (max_sse > had_sse) {
    dfree(ctx->d_sse_items);
    dfree(ctx->d_partials);
    HIP_OR_FAIL(ctx, dalloc(&ctx->d_sse_items, max_sse));
    HIP_OR_FAIL(ctx, dalloc(&ctx->d_partials, als::reduce_partials(max_sse)));
  }
  ctx->n_bins = n_bins;
  return ALS_OK;
}

als_status als_tensor_half_sweep(als_ctx *ctx, als_mode mode, float *U, float *V, float *T,
                                 float lambda, double *rmse_out) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (ctx->n_bins <= 0) return fail(ctx, ALS_ERR_INVALID_ARG, "no time bins set");
  if (mode != ALS_MODE_USERS && mode != ALS_MODE_ITEMS && mode != ALS_MODE_TIME)
    return fail(ctx, ALS_ERR_INVALID_ARG, "mode %d is not a tensor mode", (int)mode);
  if (!U || !V || !T) return fail(ctx, ALS_ERR_INVALID_ARG, "NULL factor buffer");
  if (!std::isfinite(lambda) || lambda < 0.f)
    return fail(ctx, ALS_ERR_INVALID_ARG, "lambda must be finite and >= 0");
  if (((uintptr_t)U & 15) || ((uintptr_t)V & 15) || ((uintptr_t)T & 15))
    return fail(ctx, ALS_ERR_INVALID_ARG, "factor buffers must be 16-byte aligned");
  if (ctx->d_w) return fail(ctx, ALS_ERR_INVALID_ARG, "tensor ALS takes no rating weights; detach them");
  const size_t bu = sizeof(float) * ctx->M * ctx->D, bv = sizeof(float) * ctx->N * ctx->D;
  const size_t bt = sizeof(float) * (size_t)ctx->n_bins * ctx->D;
  if (overlap(U, bu, V, bv) || overlap(U, bu, T, bt) || overlap(V, bv, T, bt))
    return fail(ctx, ALS_ERR_INVALID_ARG, "U, V and T must not overlap");
  DeviceGuard g(ctx->device);
  // the solved mode's fixed vectors are F1[idx] * F2[idx2]
  const float *F1, *F2;
  int64_t n1, n2;
  float *out;
  SweepSpec sp;
  sp.plan = (int)mode;
  if (mode == ALS_MODE_USERS) {
    F1 = V; n1 = ctx->N; F2 = T; n2 = ctx->n_bins; out = U;
    sp.idx = ctx->d_col; sp.val = ctx->d_val; sp.hd.idx2 = ctx->d_tbin;
  } else if (mode == ALS_MODE_ITEMS) {
    F1 = U; n1 = ctx->M; F2 = T; n2 = ctx->n_bins; out = V;
    sp.idx = ctx->d_row_idx; sp.val = ctx->d_val_t; sp.hd.idx2 = ctx->d_tbin_t;
  } else {
    F1 = U; n1 = ctx->M; F2 = V; n2 = ctx->N; out = T;
    sp.idx = ctx->d_tb_user; sp.val = ctx->d_tb_val; sp.hd.idx2 = ctx->d_tb_item;
  }
  sp.n_fixed = n1;
  sp.hd.Tp = ctx->d_fpad2;
  {
    PhaseTimer t(ctx, 0);
    HIP_OR_FAIL(ctx, als::launch_stage_fixed(F1, n1, ctx->D, ctx->DP, ctx->d_fpad, ctx->stream));
    HIP_OR_FAIL(ctx, als::launch_stage_fixed(F2, n2, ctx->D, ctx->DP, ctx->d_fpad2, ctx->stream));
  }
  return run_sweep(ctx, sp, lambda, out, rmse_out, als::RowPrior{});
}

als_status als_tensor_rmse(als_ctx *ctx, const float *U, const float *V, const float *T,
                           double *rmse_out) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (ctx->n_bins <= 0) return fail(ctx, ALS_ERR_INVALID_ARG, "no time bins set");
  if (!U || !V || !T || !rmse_out) return fail(ctx, ALS_ERR_INVALID_ARG, "NULL argument");
  if (((uintptr_t)U & 15) || ((uintptr_t)V & 15) || ((uintptr_t)T & 15))
    return fail(ctx, ALS_ERR_INVALID_ARG, "factor buffers must be 16-byte aligned");
  DeviceGuard g(ctx->device);
  {
    PhaseTimer t(ctx, 0);
    HIP_OR_FAIL(ctx, als::launch_stage_fixed(V, ctx->N, ctx->D, ctx->DP, ctx->d_fpad, ctx->stream));
    HIP_OR_FAIL(ctx, als::launch_stage_fixed(T, ctx->n_bins, ctx->D, ctx->DP, ctx->d_fpad2,
                                             ctx->stream));
  }
  als::Hadamard hd;
  hd.idx2 = ctx->d_tbin;
  hd.Tp = ctx->d_fpad2;
  als_status st = residual_pass(ctx, ctx->plan[ALS_ROWS_USERS], ctx->d_col, ctx->d_val, ctx->N,
                                U, hd);
  if (st != ALS_OK) return st;
  HIP_OR_FAIL(ctx, hipMemcpyAsync(ctx->h_sse, ctx->d_sse_total, sizeof(double),
                                  hipMemcpyDeviceToHost, ctx->stream));
  HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
  *rmse_out = ctx->nnz > 0 ? std::sqrt(*ctx->h_sse / (double)ctx->nnz) : 0.0;
  return ALS_OK;
}

// ---- BPTF: the tensor model's Gibbs step -------------------------------------------

als_status als_tensor_gibbs_half_sweep(als_ctx *ctx, als_mode mode, float *U, float *V, float *T,
                                       float alpha, const double *Lambda, const double *mu,
                                       const float *z, double *rmse_out) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (ctx->n_bins <= 0) return fail(ctx, ALS_ERR_INVALID_ARG, "no time bins set");
  if (mode != ALS_MODE_USERS && mode != ALS_MODE_ITEMS && mode != ALS_MODE_TIME)
    return fail(ctx, ALS_ERR_INVALID_ARG, "mode %d is not a tensor mode", (int)mode);
  if (!U || !V || !T || !Lambda || !mu || !z)
    return fail(ctx, ALS_ERR_INVALID_ARG, "NULL argument");
  if (!(alpha > 0.f) || !std::isfinite(alpha))
    return fail(ctx, ALS_ERR_INVALID_ARG, "alpha must be finite and > 0");
  if (((uintptr_t)U & 15) || ((uintptr_t)V & 15) || ((uintptr_t)T & 15))
    return fail(ctx, ALS_ERR_INVALID_ARG, "factor buffers must be 16-byte aligned");
  if (ctx->d_w) return fail(ctx, ALS_ERR_INVALID_ARG, "BPTF takes no rating weights; detach them");
  const int D = ctx->D;
  const int64_t K = ctx->n_bins;
  const size_t bu = sizeof(float) * ctx->M * D, bv = sizeof(float) * ctx->N * D;
  const size_t bt = sizeof(float) * (size_t)K * D;
  if (overlap(U, bu, V, bv) || overlap(U, bu, T, bt) || overlap(V, bv, T, bt))
    return fail(ctx, ALS_ERR_INVALID_ARG, "U, V and T must not overlap");
  const size_t bo = mode == ALS_MODE_USERS ? bu : (mode == ALS_MODE_ITEMS ? bv : bt);
  float *out = mode == ALS_MODE_USERS ? U : (mode == ALS_MODE_ITEMS ? V : T);
  if (overlap(z, bo, out, bo)) return fail(ctx, ALS_ERR_INVALID_ARG, "z overlaps the drawn factors");
  DeviceGuard g(ctx->device);
  als_status st = ensure_bayes(ctx);
  if (st != ALS_OK) return st;
  const float *F1, *F2;
  int64_t n1, n2;
  SweepSpec sp;
  sp.plan = (int)mode;
  if (mode == ALS_MODE_USERS) {
    F1 = V; n1 = ctx->N; F2 = T; n2 = K;
    sp.idx = ctx->d_col; sp.val = ctx->d_val; sp.hd.idx2 = ctx->d_tbin;
  } else if (mode == ALS_MODE_ITEMS) {
    F1 = U; n1 = ctx->M; F2 = T; n2 = K;
    sp.idx = ctx->d_row_idx; sp.val = ctx->d_val_t; sp.hd.idx2 = ctx->d_tbin_t;
  } else {
    F1 = U; n1 = ctx->M; F2 = V; n2 = ctx->N;
    sp.idx = ctx->d_tb_user; sp.val = ctx->d_tb_val; sp.hd.idx2 = ctx->d_tb_item;
  }
  sp.n_fixed = n1;
  sp.hd.Tp = ctx->d_fpad2;
  {
    PhaseTimer t(ctx, 0);
    HIP_OR_FAIL(ctx, als::launch_stage_fixed(F1, n1, D, ctx->DP, ctx->d_fpad, ctx->stream));
    HIP_OR_FAIL(ctx, als::launch_stage_fixed(F2, n2, D, ctx->DP, ctx->d_fpad2, ctx->stream));
  }
  als::RowPrior pr;
  pr.init = ctx->d_prior_init;
  pr.z = z;
  pr.zscale = (float)(1.0 / std::sqrt((double)alpha));
  if (mode != ALS_MODE_TIME) {
    HIP_OR_FAIL(ctx, als::launch_prior_prepare(Lambda, mu, D, ctx->DP, (double)alpha,
                                               !ctx->plan[mode].zero_rows.empty(),
                                               ctx->d_prior_init, ctx->d_prior_K,
                                               ctx->d_prior_mu32, ctx->d_prior_ok, ctx->stream));
    return run_sweep(ctx, sp, 0.f, out, rmse_out, pr);
  }
  // the time chain: the image is Lambda_T / alpha without a mean term; bin k takes twice
  // the image (once for its own step, once as the condition of bin k + 1), the last bin
  // once, and its neighbours' right-hand side from k_time_rhs; even bins, then odd bins
  if (!ctx->d_zero_mu) {
    st = ensure(ctx, &ctx->d_zero_mu, (size_t)D, "zero mean");
    if (st != ALS_OK) return st;
    HIP_OR_FAIL(ctx, als::launch_fill_i32(reinterpret_cast<int32_t *>(ctx->d_zero_mu), 2 * D, 0,
                                          ctx->stream));
  }
  if (ctx->time_h0_bins != K) {
    HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
    dfree(ctx->d_time_h0);
    HIP_OR_FAIL(ctx, dalloc(&ctx->d_time_h0, K * D));
    ctx->time_h0_bins = K;
  }
  HIP_OR_FAIL(ctx, als::launch_prior_prepare(Lambda, ctx->d_zero_mu, D, ctx->DP, (double)alpha,
                                             false, ctx->d_prior_init, ctx->d_prior_K,
                                             ctx->d_prior_mu32, ctx->d_prior_ok, ctx->stream));
  pr.scale = 2.f;
  pr.scale_last = 1.f;
  pr.last_row = K - 1;
  pr.h0 = ctx->d_time_h0;
  for (int parity = 0; parity < 2; ++parity) {
    HIP_OR_FAIL(ctx, als::launch_time_rhs(T, K, D, Lambda, mu, (double)alpha, parity,
                                          ctx->d_time_h0, ctx->stream));
    SweepSpec sq = sp;
    sq.plan = 3 + parity;
    sq.keep_flags = parity == 1;
    sq.sse_in_part = parity;
    st = run_sweep(ctx, sq, 0.f, T, nullptr, pr);
    if (st != ALS_OK) return st;
  }
  if (rmse_out) {
    st = als_tensor_rmse(ctx, U, V, T, rmse_out);
    if (st != ALS_OK) return st;
    if (*ctx->h_flag > 0)
      return fail(ctx, ALS_ERR_NOT_SPD, "%d time bins were flagged and left unchanged",
                  (int)*ctx->h_flag);
  }
  return ALS_OK;
}

als_status als_sample_time_hyper(als_ctx *ctx, const float *T, const double *chi2,
                                 const double *offdiag, const double *z_mu, double *mu_out,
                                 double *Lambda_out, int32_t *status_out) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (ctx->n_bins <= 0) return fail(ctx, ALS_ERR_INVALID_ARG, "no time bins set");
  if (!ctx->nw_set[2]) return fail(ctx, ALS_ERR_INVALID_ARG, "no Normal-Wishart prior set for the time chain");
  if (!T || !chi2 || (!offdiag && ctx->D > 1) || !z_mu || !mu_out || !Lambda_out)
    return fail(ctx, ALS_ERR_INVALID_ARG, "NULL argument");
  DeviceGuard g(ctx->device);
  const int64_t ntri = (int64_t)ctx->D * (ctx->D + 1) / 2;
  als_status st = ensure_bayes(ctx);
  if (st == ALS_OK) st = ensure(ctx, &ctx->d_time_extra, (size_t)ntri, "chain scatter");
  if (st != ALS_OK) return st;
  int64_t per = 0, nblk = 0;
  als::time_step_blocks(ctx->n_bins, ctx->D, per, nblk);
  if (nblk * ntri > ctx->time_partials_cap) {
    HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
    dfree(ctx->d_time_partials);
    HIP_OR_FAIL(ctx, dalloc(&ctx->d_time_partials, nblk * ntri));
    ctx->time_partials_cap = nblk * ntri;
  }
  HIP_OR_FAIL(ctx, als::launch_time_hyper(T, ctx->n_bins, ctx->D, ctx->d_nw_mu0[2],
                                          ctx->nw_beta0[2], ctx->d_nw_W0inv[2], ctx->nw_nu0[2],
                                          chi2, offdiag, z_mu, ctx->d_bayes_scratch,
                                          ctx->d_time_partials, ctx->d_time_extra, mu_out,
                                          Lambda_out, ctx->d_hyper_status, ctx->stream));
  if (status_out) {
    HIP_OR_FAIL(ctx, hipMemcpyAsync(ctx->h_hyper_status, ctx->d_hyper_status, sizeof(int32_t),
                                    hipMemcpyDeviceToHost, ctx->stream));
    HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
    *status_out = *ctx->h_hyper_status;
    if (*status_out != 0)
      return fail(ctx, ALS_ERR_NOT_SPD, "a factorisation of the Normal-Wishart draw failed");
  }
  return ALS_OK;
}

als_status als_tensor_sample_alpha(als_ctx *ctx, const float *U, const float *V, const float *T,
                                   double w0, double chi2, double *alpha_out) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (!alpha_out) return fail(ctx, ALS_ERR_INVALID_ARG, "NULL argument");
  if (!(w0 > 0.0) || !std::isfinite(w0) || !(chi2 > 0.0) || !std::isfinite(chi2))
    return fail(ctx, ALS_ERR_INVALID_ARG, "w0 and chi2 must be finite and > 0");
  double rmse = 0.0;
  als_status st = als_tensor_rmse(ctx, U, V, T, &rmse);
  if (st != ALS_OK) return st;
  *alpha_out = chi2 / (1.0 / w0 + *ctx->h_sse);
  return ALS_OK;
}

// ---- held-out predictions ----------------------------------------------------------

als_status als_predict(als_ctx *ctx, const float *U, const float *V, int64_t n_pairs,
                       const int32_t *users, const int32_t *items, float *pred) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (n_pairs < 0 || n_pairs > kMaxPairs)
    return fail(ctx, ALS_ERR_INVALID_ARG, "n_pairs out of range");
  if (n_pairs == 0) return ALS_OK;
  if (!U || !V || !users || !items || !pred) return fail(ctx, ALS_ERR_INVALID_ARG, "NULL argument");
  if (((uintptr_t)U & 15) || ((uintptr_t)V & 15))
    return fail(ctx, ALS_ERR_INVALID_ARG, "factor buffers must be 16-byte aligned");
  const size_t pb = sizeof(float) * (size_t)n_pairs;
  if (overlap(pred, pb, U, sizeof(float) * ctx->M * ctx->D) ||
      overlap(pred, pb, V, sizeof(float) * ctx->N * ctx->D) ||
      overlap(pred, pb, users, sizeof(int32_t) * n_pairs) ||
      overlap(pred, pb, items, sizeof(int32_t) * n_pairs))
    return fail(ctx, ALS_ERR_INVALID_ARG, "pred overlaps an input");
  DeviceGuard g(ctx->device);
  HIP_OR_FAIL(ctx, als::launch_predict(U, V, ctx->M, ctx->N, ctx->D, n_pairs, users, items,
                                       nullptr, pred, nullptr, ctx->stream));
  return ALS_OK;
}

als_status als_set_holdout(als_ctx *ctx, int64_t n_pairs, const int32_t *users,
                           const int32_t *items, const uint8_t *ratings) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (n_pairs < 0 || n_pairs > kMaxPairs)
    return fail(ctx, ALS_ERR_INVALID_ARG, "n_pairs out of range");
  if (n_pairs > 0 && (!users || !items || !ratings))
    return fail(ctx, ALS_ERR_INVALID_ARG, "NULL argument");
  for (int64_t p = 0; p < n_pairs; ++p) {
    if (users[p] < 0 || users[p] >= ctx->M || items[p] < 0 || items[p] >= ctx->N)
      return fail(ctx, ALS_ERR_INVALID_ARG, "pair %lld: (%d, %d) outside %lld x %lld",
                  (long long)p, users[p], items[p], (long long)ctx->M, (long long)ctx->N);
  }
  DeviceGuard g(ctx->device);
  HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
  free_holdout(ctx);
  if (n_pairs == 0) {
    ctx->n_hold = 0;
    return ALS_OK;
  }
  // counting sort by user, stable: pairs of one user become adjacent (their u rows are
  // then read once from memory), in the caller's order within a user
  std::vector<int64_t> start(ctx->M + 1, 0);
  for (int64_t p = 0; p < n_pairs; ++p) start[users[p] + 1] += 1;
  for (int64_t u = 0; u < ctx->M; ++u) start[u + 1] += start[u];
  std::vector<int32_t> hu(n_pairs), hi(n_pairs);
  std::vector<uint8_t> hr(n_pairs);
  for (int64_t p = 0; p < n_pairs; ++p) {
    const int64_t q = start[users[p]]++;
    hu[q] = users[p];
    hi[q] = items[p];
    hr[q] = ratings[p];
  }
  const int64_t nb = als::pair_blocks(n_pairs, ctx->D);
  hipError_t e = dalloc(&ctx->d_hu, n_pairs);
  if (e == hipSuccess) e = dalloc(&ctx->d_hi, n_pairs);
  if (e == hipSuccess) e = dalloc(&ctx->d_hr, n_pairs);
  if (e == hipSuccess) e = dalloc(&ctx->d_hold_blocks, nb);
  if (e == hipSuccess) e = dalloc(&ctx->d_hold_partials, als::reduce_partials(nb));
  if (e == hipSuccess) e = dalloc(&ctx->d_hold_sse, 1);
  if (e == hipSuccess)
    e = hipMemcpy(ctx->d_hu, hu.data(), sizeof(int32_t) * n_pairs, hipMemcpyHostToDevice);
  if (e == hipSuccess)
    e = hipMemcpy(ctx->d_hi, hi.data(), sizeof(int32_t) * n_pairs, hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(ctx->d_hr, hr.data(), n_pairs, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    free_holdout(ctx);
    return fail(ctx, e == hipErrorOutOfMemory ? ALS_ERR_OUT_OF_MEMORY : ALS_ERR_HIP,
                "held-out pairs: %s", hipGetErrorString(e));
  }
  ctx->n_hold = n_pairs;
  return ALS_OK;
}

als_status als_holdout_rmse(als_ctx *ctx, const float *U, const float *V, double *rmse_out) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (!U || !V || !rmse_out) return fail(ctx, ALS_ERR_INVALID_ARG, "NULL argument");
  if (ctx->n_hold < 0) return fail(ctx, ALS_ERR_INVALID_ARG, "no held-out pairs registered");
  if (((uintptr_t)U & 15) || ((uintptr_t)V & 15))
    return fail(ctx, ALS_ERR_INVALID_ARG, "factor buffers must be 16-byte aligned");
  if (ctx->n_hold == 0) {
    *rmse_out = 0.0;
    return ALS_OK;
  }
  DeviceGuard g(ctx->device);
  HIP_OR_FAIL(ctx, als::launch_predict(U, V, ctx->M, ctx->N, ctx->D, ctx->n_hold, ctx->d_hu,
                                       ctx->d_hi, ctx->d_hr, nullptr, ctx->d_hold_blocks,
                                       ctx->stream));
  HIP_OR_FAIL(ctx, als::launch_reduce(ctx->d_hold_blocks, als::pair_blocks(ctx->n_hold, ctx->D),
                                      ctx->d_hold_partials, ctx->d_hold_sse, ctx->stream));
  HIP_OR_FAIL(ctx, hipMemcpyAsync(ctx->h_sse, ctx->d_hold_sse, sizeof(double),
                                  hipMemcpyDeviceToHost, ctx->stream));
  HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
  *rmse_out = std::sqrt(*ctx->h_sse / (double)ctx->n_hold);
  return ALS_OK;
}

als_status als_pair_rmse_noalloc(als_ctx *ctx, const float *U, const float *V, int64_t n_pairs,
                                 const int32_t *users, const int32_t *items,
                                 const uint8_t *ratings, double *rmse_out) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  ctx->err.clear();
  if (!U || !V || !rmse_out) return fail(ctx, ALS_ERR_INVALID_ARG, "NULL argument");
  if (n_pairs < 0 || n_pairs > kNoAllocMaxPairs)
    return fail(ctx, ALS_ERR_INVALID_ARG,
                "n_pairs = %lld outside [0, %lld], the capacity of the fixed scratch array",
                (long long)n_pairs, (long long)kNoAllocMaxPairs);
  if (n_pairs > 0 && (!users || !items || !ratings))
    return fail(ctx, ALS_ERR_INVALID_ARG, "NULL pair array");
  if (((uintptr_t)U & 15) || ((uintptr_t)V & 15))
    return fail(ctx, ALS_ERR_INVALID_ARG, "factor buffers must be 16-byte aligned");
  if (n_pairs == 0) {
    *rmse_out = 0.0;
    return ALS_OK;
  }
  // scratch layout: per-block squared errors [nb], the reduction's partials [np], total [1]
  const int64_t nb = als::pair_blocks(n_pairs, ctx->D);
  const int64_t np = als::reduce_partials(nb);
  if (nb + np + 1 > kScratchDoubles)
    return fail(ctx, ALS_ERR_INVALID_ARG, "%lld pairs need %lld scratch doubles, above %lld",
                (long long)n_pairs, (long long)(nb + np + 1), (long long)kScratchDoubles);
  DeviceGuard g(ctx->device);
  double *blocks = ctx->d_scratch, *partials = blocks + nb, *total = partials + np;
  HIP_OR_FAIL(ctx, als::launch_predict(U, V, ctx->M, ctx->N, ctx->D, n_pairs, users, items,
                                       ratings, nullptr, blocks, ctx->stream));
  HIP_OR_FAIL(ctx, als::launch_reduce(blocks, nb, partials, total, ctx->stream));
  HIP_OR_FAIL(ctx, hipMemcpyAsync(ctx->h_sse, total, sizeof(double), hipMemcpyDeviceToHost,
                                  ctx->stream));
  HIP_OR_FAIL(ctx, hipStreamSynchronize(ctx->stream));
  *rmse_out = std::sqrt(*ctx->h_sse / (double)n_pairs);
  return ALS_OK;
}

als_status als_set_profiling(als_ctx *ctx, int32_t enable) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  if (enable < 0 || enable > 2)
    return fail(ctx, ALS_ERR_INVALID_ARG, "profiling mode %d is not 0, 1 or 2", (int)enable);
  als_status st = collect_profile(ctx);
  if (st != ALS_OK) return st;
  ctx->profiling = enable != 0;
  ctx->prof_mode = enable;
  if (enable) {
    for (int i = 0; i < kPhases; ++i) {
      ctx->prof_ms[i] = 0.0;
      ctx->prof_n[i] = 0;
    }
  }
  return ALS_OK;
}

als_status als_get_profile(als_ctx *ctx, int32_t phase, double *total_ms, int64_t *launches) {
  if (!ctx) return fail(nullptr, ALS_ERR_INVALID_ARG, "NULL context");
  if (phase < 0 || phase >= kPhases || !total_ms || !launches)
    return fail(ctx, ALS_ERR_INVALID_ARG, "bad argument");
  als_status st = collect_profile(ctx);
  if (st != ALS_OK) return st;
  *total_ms = ctx->prof_ms[phase];
  *launches = ctx->prof_n[phase];
  return ALS_OK;
}

void als_destroy(als_ctx *ctx) {
  if (!ctx) return;
  {
    DeviceGuard g(ctx->device);
    (void)hipStreamSynchronize(ctx->stream);
  }
  free_ctx(ctx);
}

}  // extern "C"
