// Partial normal equations of the ALS row update (Sec. 2.2) on fp32 MFMA.
//
// For a work item (a row, or a chunk of a split row) with ratings k, fixed
// rows f_k (width D) and ratings r_k, one wavefront accumulates
//     G = sum_k f_k f_k^T   (upper-triangle 16x16 tiles only)
//     b = sum_k r_k f_k
// and stores them into the item's workspace slot. The Gram build is the
// dense contraction F^T F over the item's ratings, so it runs on
// v_mfma_f32_16x16x4f32: one MFMA consumes four ratings; lane (k, c)
// (k = lane / 16, c = lane % 16) supplies feature 16*I + c of rating k for
// block I, and the same register is both operands of a diagonal tile.
// The width is padded to DP = 16 * ceil(D / 16) with zero features.
//
// Ratings are processed in groups of 64: one coalesced load brings the 64
// column indices and ratings (prefetched one group ahead), and lanes fetch the
// index of their step's rating with a cross-lane permute. The feature loads
// of STEPS steps are issued before their MFMAs to keep memory requests in
// flight.
#include "internal.h"

namespace als {

typedef float floatx4 __attribute__((ext_vector_type(4)));

template <int DP>
struct GramCfg {
  static constexpr int T = DP / 16;
  static constexpr int NT = T * (T + 1) / 2;
  // steps (of four ratings) whose feature loads are issued together
  static constexpr int STEPS = T <= 2 ? 16 : (T <= 4 ? 8 : 4);
};

template <int DP>
__global__ __launch_bounds__(64) void k_gram(const WorkItem *__restrict__ items,
                                             const int32_t *__restrict__ idx,
                                             const uint8_t *__restrict__ val,
                                             const float *__restrict__ F, int D,
                                             float *__restrict__ ws) {
  using C = GramCfg<DP>;
  constexpr int T = C::T, NT = C::NT, STEPS = C::STEPS;
  const WorkItem it = items[blockIdx.x];
  const int lane = threadIdx.x;
  const int kq = lane >> 4;  // rating within a step
  const int c = lane & 15;   // feature within a block
  const int n = it.len;
  const int32_t *__restrict__ ip = idx + it.start;
  const uint8_t *__restrict__ vp = val + it.start;

  bool colok[T];
#pragma unroll
  for (int I = 0; I < T; ++I) colok[I] = 16 * I + c < D;

  floatx4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  float rhs[T];
#pragma unroll
  for (int I = 0; I < T; ++I) rhs[I] = 0.f;

  // group of 64 ratings: lane l holds index and rating of rating g*64 + l
  int jv = lane < n ? ip[lane] : 0;
  float rv = lane < n ? (float)vp[lane] : 0.f;

  for (int g = 0; g < n; g += 64) {
    const int gn = g + 64 + lane;
    const int jn = gn < n ? ip[gn] : 0;
    const float rn = gn < n ? (float)vp[gn] : 0.f;
    const int steps = min(16, (n - g + 3) >> 2);
#pragma unroll
    for (int s0 = 0; s0 < 16; s0 += STEPS) {
      if (s0 >= steps) break;
      float a[STEPS][T];
      float r[STEPS];
#pragma unroll
      for (int u = 0; u < STEPS; ++u) {
        const int src = 4 * (s0 + u) + kq;
        const int j = __shfl(jv, src);
        r[u] = __shfl(rv, src);
        const bool ok = g + src < n;
        const float *__restrict__ fr = F + (int64_t)j * D + c;
#pragma unroll
        for (int I = 0; I < T; ++I) a[u][I] = (ok && colok[I]) ? fr[16 * I] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < STEPS; ++u) {
        if (s0 + u < steps) {
#pragma unroll
          for (int I = 0; I < T; ++I) rhs[I] = fmaf(r[u], a[u][I], rhs[I]);
          int t = 0;
#pragma unroll
          for (int I = 0; I < T; ++I) {
#pragma unroll
            for (int J = I; J < T; ++J) {
              acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u][I], a[u][J], acc[t], 0, 0, 0);
              ++t;
            }
          }
        }
      }
    }
    jv = jn;
    rv = rn;
  }

  // the four rating groups of a lane column hold partial right-hand sides
#pragma unroll
  for (int I = 0; I < T; ++I) {
    rhs[I] += __shfl_xor(rhs[I], 16);
    rhs[I] += __shfl_xor(rhs[I], 32);
  }
  float *__restrict__ out = ws + it.slot * (int64_t)slot_floats(DP);
#pragma unroll
  for (int t = 0; t < NT; ++t) *reinterpret_cast<floatx4 *>(out + t * 256 + lane * 4) = acc[t];
  if (kq == 0) {
#pragma unroll
    for (int I = 0; I < T; ++I) out[NT * 256 + 16 * I + c] = rhs[I];
  }
}

template <int DP>
static hipError_t launch_gram_t(const WorkItem *items, int64_t n_items, const int32_t *idx,
                                const uint8_t *val, const float *F, int D, float *ws,
                                hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_gram<DP>, dim3((unsigned)n_items), dim3(64), 0, s, items, idx, val, F, D,
                     ws);
  return hipGetLastError();
}

hipError_t launch_gram(int dp, const WorkItem *items, int64_t n_items, const int32_t *idx,
                       const uint8_t *val, const float *F, int D, float *ws, hipStream_t s) {
  switch (dp) {
    case 16: return launch_gram_t<16>(items, n_items, idx, val, F, D, ws, s);
    case 32: return launch_gram_t<32>(items, n_items, idx, val, F, D, ws, s);
    case 48: return launch_gram_t<48>(items, n_items, idx, val, F, D, ws, s);
    case 64: return launch_gram_t<64>(items, n_items, idx, val, F, D, ws, s);
    case 80: return launch_gram_t<80>(items, n_items, idx, val, F, D, ws, s);
    case 96: return launch_gram_t<96>(items, n_items, idx, val, F, D, ws, s);
    case 112: return launch_gram_t<112>(items, n_items, idx, val, F, D, ws, s);
    case 128: return launch_gram_t<128>(items, n_items, idx, val, F, D, ws, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace als
