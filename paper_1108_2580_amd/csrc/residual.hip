// Residuals of the predictions r_hat = x_s . f_j (Sec. 2.2) of a given state,
// for the training RMSE of Sec. 4.1 (the standalone pass behind als_rmse and
// the new-state RMSE of als_half_sweep). One wavefront per work item (row or
// chunk of a split row); each lane takes whole ratings: it gathers the staged
// fixed row f_j (row stride DP, 16-byte aligned, zero padded) with float4
// loads, forms the dot product with x_s (held in LDS), and accumulates
// (r - x_s . f_j)^2 in fp64. The wavefront total goes to sse_items[item]; a
// fixed-order reduction over items follows. TS (tensor ALS): f is the elementwise
// product of the staged rows Fp[j] and hd.Tp[t], t the rating's second index.
#include "internal.h"

namespace als {

template <int DP, bool TS>
__global__ __launch_bounds__(64) void k_resid(const WorkItem *__restrict__ items,
                                              const int32_t *__restrict__ idx,
                                              const uint8_t *__restrict__ val,
                                              const float *__restrict__ Fp,
                                              const float *__restrict__ X, int D,
                                              double *__restrict__ sse_items, Hadamard hd) {
  __shared__ float xs[DP];
  const WorkItem it = items[blockIdx.x];
  const int lane = threadIdx.x;
  for (int d = lane; d < DP; d += 64) xs[d] = d < D ? X[(int64_t)it.row * D + d] : 0.f;
  __syncthreads();
  const int32_t *__restrict__ ip = idx + it.start;
  const uint8_t *__restrict__ vp = val + it.start;
  const int D4 = (D + 3) >> 2;
  double acc = 0.0;
  for (int q = lane; q < it.len; q += 64) {
    const float4 *__restrict__ f = reinterpret_cast<const float4 *>(Fp + (int64_t)ip[q] * DP);
    const float4 *__restrict__ h =
        TS ? reinterpret_cast<const float4 *>(hd.Tp + (int64_t)hd.idx2[it.start + q] * DP)
           : nullptr;
    float dot = 0.f;
#pragma unroll
    for (int d4 = 0; d4 < DP / 4; ++d4) {
      if (d4 < D4) {
        float4 v = f[d4];
        if constexpr (TS) {
          const float4 t = h[d4];
          v.x *= t.x;
          v.y *= t.y;
          v.z *= t.z;
          v.w *= t.w;
        }
        dot = fmaf(v.x, xs[4 * d4 + 0], dot);
        dot = fmaf(v.y, xs[4 * d4 + 1], dot);
        dot = fmaf(v.z, xs[4 * d4 + 2], dot);
        dot = fmaf(v.w, xs[4 * d4 + 3], dot);
      }
    }
    const double e = (double)vp[q] - (double)dot;
    acc = fma(e, e, acc);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if (lane == 0) sse_items[blockIdx.x] = acc;
}

template <int DP>
static hipError_t launch_resid_t(const WorkItem *items, int64_t n_items, const int32_t *idx,
                                 const uint8_t *val, const float *Fp, const float *X, int D,
                                 double *sse_items, const Hadamard &hd, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  if (hd.idx2)
    hipLaunchKernelGGL((k_resid<DP, true>), dim3((unsigned)n_items), dim3(64), 0, s, items, idx,
                       val, Fp, X, D, sse_items, hd);
  else
    hipLaunchKernelGGL((k_resid<DP, false>), dim3((unsigned)n_items), dim3(64), 0, s, items, idx,
                       val, Fp, X, D, sse_items, hd);
  return hipGetLastError();
}

hipError_t launch_resid(int dp, const WorkItem *items, int64_t n_items, const int32_t *idx,
                        const uint8_t *val, const float *Fp, const float *X, int D,
                        double *sse_items, const Hadamard &hd, hipStream_t s) {
  switch (dp) {
    case 16: return launch_resid_t<16>(items, n_items, idx, val, Fp, X, D, sse_items, hd, s);
    case 32: return launch_resid_t<32>(items, n_items, idx, val, Fp, X, D, sse_items, hd, s);
    case 48: return launch_resid_t<48>(items, n_items, idx, val, Fp, X, D, sse_items, hd, s);
    case 64: return launch_resid_t<64>(items, n_items, idx, val, Fp, X, D, sse_items, hd, s);
    case 80: return launch_resid_t<80>(items, n_items, idx, val, Fp, X, D, sse_items, hd, s);
    case 96: return launch_resid_t<96>(items, n_items, idx, val, Fp, X, D, sse_items, hd, s);
    case 112: return launch_resid_t<112>(items, n_items, idx, val, Fp, X, D, sse_items, hd, s);
    case 128: return launch_resid_t<128>(items, n_items, idx, val, Fp, X, D, sse_items, hd, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace als
