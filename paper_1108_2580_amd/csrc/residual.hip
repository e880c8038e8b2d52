// Residuals of the predictions r_hat = x_s . f_j (Sec. 2.2) of a given state, for the
// training RMSE of Sec. 4.1 (the standalone pass behind als_rmse, als_tensor_rmse, the
// new-state RMSE of a half-sweep, and the rating-precision draw of BPTF).
//
// One wavefront per work item (row, or chunk of a split row), with the gather of the
// Gram kernels (gram.h): a 64-rating group is staged in LDS, and lane (kq, c) loads
// feature 16 X + c of the staged fixed row of rating 4 s + kq for all 16 steps s of the
// group at once, so that every load instruction reads four rows in contiguous 64-byte
// segments. Lane (kq, c) forms the per-step partial dot products with its features of
// x_s; the group's 16 x 16 partials are summed over the feature lanes through an LDS
// transpose (group_residuals), after which each lane holds one rating's prediction and
// adds (r - r_hat)^2 in fp64.
// The wavefront total goes to sse_items[item]; a fixed-order reduction over the items
// follows. TS (tensor ALS): f is the elementwise product of the staged rows Fp[j] and
// hd.Tp[t], t the rating's second index.
#include "gram.h"

namespace als {

template <int DP, bool TS>
__global__ __launch_bounds__(64) void k_resid(const WorkItem *__restrict__ items,
                                              const int32_t *__restrict__ idx,
                                              const uint8_t *__restrict__ val,
                                              const float *__restrict__ Fp, int zrow,
                                              const float *__restrict__ X, int D,
                                              double *__restrict__ sse_items, Hadamard hd) {
  constexpr int T = DP / 16;
  __shared__ GroupStage st;
  const WorkItem it = items[blockIdx.x];
  const int lane = threadIdx.x, c = lane & 15;
  float xo[T];
#pragma unroll
  for (int Xt = 0; Xt < T; ++Xt) {
    const float v = X[(int64_t)it.row * D + min(16 * Xt + c, D - 1)];
    xo[Xt] = 16 * Xt + c < D ? v : 0.f;
  }
  const int32_t *__restrict__ ip = idx + it.start;
  const uint8_t *__restrict__ vp = val + it.start;
  const int32_t *__restrict__ tp = TS ? hd.idx2 + it.start : nullptr;
  const int n = it.len;
  GroupLanes gv = first_group<false, TS>(ip, vp, nullptr, tp, n, zrow);
  double sse = 0.0;
  for (int g = 0; g < n; g += 64) {
    const GroupLanes gn = group_lanes<false, TS>(ip, vp, nullptr, tp, n, g + 64, zrow);
    stage_group<false, TS>(st, 0, gv);
    wave_sync();
    float a[16][T], sb[16], r[16], w[16];
    gather_block<DP, 16, false, false, TS>(a, sb, r, w, st, 0, 0, Fp, hd.Tp, false);
    float pi[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      float t = 0.f;
#pragma unroll
      for (int Xt = 0; Xt < T; ++Xt) t = fmaf(a[u][Xt], xo[Xt], t);
      pi[u] = t;
    }
    group_residuals(pi, st, 0, g, n, sse);
    wave_sync();  // the buffer is restaged by the next group
    gv = gn;
  }
  sse = sum_wave_f64(sse);
  if (lane == 0) sse_items[blockIdx.x] = sse;
}

template <int DP>
static hipError_t launch_resid_t(const WorkItem *items, int64_t n_items, const int32_t *idx,
                                 const uint8_t *val, const float *Fp, int zrow, const float *X,
                                 int D, double *sse_items, const Hadamard &hd, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  if (hd.idx2)
    hipLaunchKernelGGL((k_resid<DP, true>), dim3((unsigned)n_items), dim3(64), 0, s, items, idx,
                       val, Fp, zrow, X, D, sse_items, hd);
  else
    hipLaunchKernelGGL((k_resid<DP, false>), dim3((unsigned)n_items), dim3(64), 0, s, items, idx,
                       val, Fp, zrow, X, D, sse_items, hd);
  return hipGetLastError();
}

hipError_t launch_resid(int dp, const WorkItem *items, int64_t n_items, const int32_t *idx,
                        const uint8_t *val, const float *Fp, int64_t n_fixed, const float *X,
                        int D, double *sse_items, const Hadamard &hd, hipStream_t s) {
  const int zrow = (int)n_fixed;
  switch (dp) {
    case 16: return launch_resid_t<16>(items, n_items, idx, val, Fp, zrow, X, D, sse_items, hd, s);
    case 32: return launch_resid_t<32>(items, n_items, idx, val, Fp, zrow, X, D, sse_items, hd, s);
    case 48: return launch_resid_t<48>(items, n_items, idx, val, Fp, zrow, X, D, sse_items, hd, s);
    case 64: return launch_resid_t<64>(items, n_items, idx, val, Fp, zrow, X, D, sse_items, hd, s);
    case 80: return launch_resid_t<80>(items, n_items, idx, val, Fp, zrow, X, D, sse_items, hd, s);
    case 96: return launch_resid_t<96>(items, n_items, idx, val, Fp, zrow, X, D, sse_items, hd, s);
    case 112: return launch_resid_t<112>(items, n_items, idx, val, Fp, zrow, X, D, sse_items, hd, s);
    case 128: return launch_resid_t<128>(items, n_items, idx, val, Fp, zrow, X, D, sse_items, hd, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace als
