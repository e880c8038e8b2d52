// Held-out predictions r_hat = u_u . v_i (Sec. 2.2) and the squared errors of
// the validation RMSE (Sec. 4.1), for a list of (user, item) pairs.
//
// The work is two gathered D-vectors and one dot product per pair, so it is
// bound by memory. Narrow or unaligned rows: one lane takes one whole pair and
// reads both rows with the widest loads their alignment allows (float4 when
// D % 4 == 0, then float2, then float), eight vectors per row in flight before
// any arithmetic. Rows of 16 floats and more (D % 4 == 0): a group of 4 or 8
// lanes shares a pair, so that each load instruction reads contiguous row
// segments (the wave's 64 lanes touch 16 or 8 rows instead of 64), and the
// group's partial sums are added by shuffles. The dot
// product runs with fused multiply-adds in fp32 (in feature order for one lane per
// pair; strided per lane, then a shuffle tree, for a group). Pairs whose
// indices fall outside the factor tables give NaN and read nothing. With
// ratings, each 256-lane block writes the fp64 sum of its pairs' squared
// errors; a fixed-order reduction follows, so the sum is reproducible.
#include "internal.h"

namespace als {

namespace {

constexpr int kPairBlock = 256;
constexpr int kVecInFlight = 8;

template <int VW> struct Vec;
template <> struct Vec<4> {
  using T = float4;
  static __device__ __forceinline__ float fma_dot(T a, T b, float acc) {
    acc = fmaf(a.x, b.x, acc);
    acc = fmaf(a.y, b.y, acc);
    acc = fmaf(a.z, b.z, acc);
    return fmaf(a.w, b.w, acc);
  }
};
template <> struct Vec<2> {
  using T = float2;
  static __device__ __forceinline__ float fma_dot(T a, T b, float acc) {
    acc = fmaf(a.x, b.x, acc);
    return fmaf(a.y, b.y, acc);
  }
};
template <> struct Vec<1> {
  using T = float;
  static __device__ __forceinline__ float fma_dot(T a, T b, float acc) { return fmaf(a, b, acc); }
};

// u . v over D features (D % VW == 0, both rows VW * 4-byte aligned), in feature order.
template <int VW>
__device__ __forceinline__ float row_dot(const float *__restrict__ u, const float *__restrict__ v,
                                         int D) {
  using T = typename Vec<VW>::T;
  const T *__restrict__ a = reinterpret_cast<const T *>(u);
  const T *__restrict__ b = reinterpret_cast<const T *>(v);
  const int nv = D / VW;
  float acc = 0.f;
  for (int c = 0; c < nv; c += kVecInFlight) {
    T x[kVecInFlight], y[kVecInFlight];
#pragma unroll
    for (int k = 0; k < kVecInFlight; ++k) {
      if (c + k < nv) {
        x[k] = a[c + k];
        y[k] = b[c + k];
      }
    }
#pragma unroll
    for (int k = 0; k < kVecInFlight; ++k)
      if (c + k < nv) acc = Vec<VW>::fma_dot(x[k], y[k], acc);
  }
  return acc;
}

// G lanes share a pair (G a power of two, 1 < G <= 16, D % 4 == 0): lane g of the group
// loads vectors g, g + G, ... of both rows, so that one load instruction of the wave reads
// whole contiguous row segments; the G partial sums are then added across the group.
template <int G, bool SSE>
__global__ __launch_bounds__(kPairBlock) void k_predict_group(
    const float *__restrict__ U, const float *__restrict__ V, int64_t M, int64_t N, int D,
    int64_t n, const int32_t *__restrict__ users, const int32_t *__restrict__ items,
    const uint8_t *__restrict__ r, float *__restrict__ pred, double *__restrict__ sse_blocks) {
  const int g = (int)threadIdx.x & (G - 1);
  const int64_t p = ((int64_t)blockIdx.x * kPairBlock + threadIdx.x) / G;
  double e2 = 0.0;
  float acc = 0.f;
  bool ok = false;
  double rv = 0.0;
  if (p < n) {
    const uint32_t u = (uint32_t)users[p], i = (uint32_t)items[p];
    rv = SSE ? (double)r[p] : 0.0;
    ok = ((uint64_t)u < (uint64_t)M) & ((uint64_t)i < (uint64_t)N);
    if (ok) {
      const float4 *__restrict__ a = reinterpret_cast<const float4 *>(U + (int64_t)u * D);
      const float4 *__restrict__ b = reinterpret_cast<const float4 *>(V + (int64_t)i * D);
      const int nv = D / 4;
      constexpr int kIn = 4;  // vectors of each row in flight per lane
      for (int c0 = g; c0 < nv; c0 += kIn * G) {
        float4 x[kIn], y[kIn];
#pragma unroll
        for (int k = 0; k < kIn; ++k) {
          if (c0 + k * G < nv) {
            x[k] = a[c0 + k * G];
            y[k] = b[c0 + k * G];
          }
        }
#pragma unroll
        for (int k = 0; k < kIn; ++k)
          if (c0 + k * G < nv) acc = Vec<4>::fma_dot(x[k], y[k], acc);
      }
    }
  }
#pragma unroll
  for (int o = G / 2; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  if (p < n && g == 0) {
    const float dot = ok ? acc : __builtin_nanf("");
    if (pred) pred[p] = dot;
    if (SSE) {
      const double e = rv - (double)dot;
      e2 = e * e;
    }
  }
  if (SSE) {
    __shared__ double wsum[kPairBlock / 64];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) e2 += __shfl_xor(e2, o);
    if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = e2;
    __syncthreads();
    if (threadIdx.x == 0) {
      double s = 0.0;
#pragma unroll
      for (int w = 0; w < kPairBlock / 64; ++w) s += wsum[w];
      sse_blocks[blockIdx.x] = s;
    }
  }
}

template <int VW, bool SSE>
__global__ __launch_bounds__(kPairBlock) void k_predict(
    const float *__restrict__ U, const float *__restrict__ V, int64_t M, int64_t N, int D,
    int64_t n, const int32_t *__restrict__ users, const int32_t *__restrict__ items,
    const uint8_t *__restrict__ r, float *__restrict__ pred, double *__restrict__ sse_blocks) {
  const int64_t p = (int64_t)blockIdx.x * kPairBlock + threadIdx.x;
  double e2 = 0.0;
  if (p < n) {
    // both indices (and the rating) are loaded before either is tested, so the two
    // index loads overlap; a negative index wraps to a large unsigned value
    const uint32_t u = (uint32_t)users[p], i = (uint32_t)items[p];
    const double rv = SSE ? (double)r[p] : 0.0;
    float dot = __builtin_nanf("");
    if (((uint64_t)u < (uint64_t)M) & ((uint64_t)i < (uint64_t)N))
      dot = row_dot<VW>(U + (int64_t)u * D, V + (int64_t)i * D, D);
    if (pred) pred[p] = dot;
    if (SSE) {
      const double e = rv - (double)dot;
      e2 = e * e;
    }
  }
  if (SSE) {
    __shared__ double wsum[kPairBlock / 64];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) e2 += __shfl_xor(e2, o);
    if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = e2;
    __syncthreads();
    if (threadIdx.x == 0) {
      double s = 0.0;
#pragma unroll
      for (int w = 0; w < kPairBlock / 64; ++w) s += wsum[w];
      sse_blocks[blockIdx.x] = s;
    }
  }
}

template <int G>
hipError_t launch_predict_group(const float *U, const float *V, int64_t M, int64_t N, int D,
                                int64_t n, const int32_t *users, const int32_t *items,
                                const uint8_t *r, float *pred, double *sse_blocks,
                                hipStream_t s) {
  const unsigned blocks = (unsigned)pair_blocks(n, D);
  if (sse_blocks)
    hipLaunchKernelGGL((k_predict_group<G, true>), dim3(blocks), dim3(kPairBlock), 0, s, U, V, M,
                       N, D, n, users, items, r, pred, sse_blocks);
  else
    hipLaunchKernelGGL((k_predict_group<G, false>), dim3(blocks), dim3(kPairBlock), 0, s, U, V, M,
                       N, D, n, users, items, r, pred, sse_blocks);
  return hipGetLastError();
}

template <int VW>
hipError_t launch_predict_vw(const float *U, const float *V, int64_t M, int64_t N, int D,
                             int64_t n, const int32_t *users, const int32_t *items,
                             const uint8_t *r, float *pred, double *sse_blocks, hipStream_t s) {
  const unsigned blocks = (unsigned)pair_blocks(n, D);
  if (sse_blocks)
    hipLaunchKernelGGL((k_predict<VW, true>), dim3(blocks), dim3(kPairBlock), 0, s, U, V, M, N, D,
                       n, users, items, r, pred, sse_blocks);
  else
    hipLaunchKernelGGL((k_predict<VW, false>), dim3(blocks), dim3(kPairBlock), 0, s, U, V, M, N,
                       D, n, users, items, r, pred, sse_blocks);
  return hipGetLastError();
}

}  // namespace

// Lanes per pair (measured on the full-size workload's pairs): rows of 96 floats and
// more (multiples of 4) take 8 lanes, rows of 16 to 92 floats 4 lanes, the rest one.
static int predict_group(int D) {
  if (D % 4 != 0) return 1;
  const int nv = D / 4;
  return nv >= 24 ? 8 : (nv >= 4 ? 4 : 1);
}

int64_t pair_blocks(int64_t n, int D) {
  return (n * predict_group(D) + kPairBlock - 1) / kPairBlock;
}

hipError_t launch_predict(const float *U, const float *V, int64_t M, int64_t N, int D, int64_t n,
                          const int32_t *users, const int32_t *items, const uint8_t *r,
                          float *pred, double *sse_blocks, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  if (pair_blocks(n, D) > 0x7fffffff || (sse_blocks && !r)) return hipErrorInvalidValue;
  const int G = predict_group(D);
  if (G == 8) return launch_predict_group<8>(U, V, M, N, D, n, users, items, r, pred, sse_blocks, s);
  if (G == 4) return launch_predict_group<4>(U, V, M, N, D, n, users, items, r, pred, sse_blocks, s);
  if (D % 4 == 0) return launch_predict_vw<4>(U, V, M, N, D, n, users, items, r, pred, sse_blocks, s);
  if (D % 2 == 0) return launch_predict_vw<2>(U, V, M, N, D, n, users, items, r, pred, sse_blocks, s);
  return launch_predict_vw<1>(U, V, M, N, D, n, users, items, r, pred, sse_blocks, s);
}

}  // namespace als
