// Narrow factor widths (D <= 20): normal equations built by the MFMA gather
// kernel, solved one row per lane.
//
// For small D a wavefront-wide factorisation leaves most lanes idle, while a
// whole D x D system fits in one lane's registers. The half-sweep therefore
// splits in two launches:
//   k_gram_ne    one wavefront per row (or chunk of a split row) accumulates
//                G = sum f f^T and b = sum r f on MFMA (gram.h), plus the
//                entering-state squared residuals, and stores the upper
//                triangle of G and b as a packed record;
//   k_sum_records sums the chunk records of each split row into its record;
//   k_solve_lane one lane per row loads its record, adds lambda * n_s to the
//                diagonal, factors
//                A = U^T U in registers, solves U^T y = b and U x = y
//                (Sec. 2.2; the per-update inversion of Sec. 4.1) and
//                writes x unless a pivot is not positive and finite. In a Gibbs
//                half-sweep (BAYES) the record gets the prior image added instead
//                (Lambda / alpha and Lambda mu / alpha), and y gets z / sqrt(alpha)
//                before the back substitution, which turns the solve into the
//                conditional draw mu* + L*^{-T} z. The time chain of BPTF scales the
//                image per row and adds a per-row right-hand side (RowPrior).
// Records hold LD(LD+1)/2 + LD floats (LD = 16 or 20, the width the solve is
// compiled for; padded features solve to zero), rounded up to a multiple of 4.
#include "gram.h"

namespace als {

// AUG (used for D = 17..20, LD = 20): the ratings ride in padding feature 20 of the
// gathered rows, so the MFMA Gram delivers b in column 20 (tile column 4 of the last
// tile) and the per-rating right-hand-side FMAs disappear. WT: weighted ALS, with the
// per-rating weights wts aligned with idx / val. TS: tensor ALS, whose fixed vectors are
// the elementwise products Fp[idx] * hd.Tp[hd.idx2].
// Waves per SIMD: six for plain ALS (under 80 registers), five for weighted and four for
// tensor ALS, which gather more per rating; the bound keeps the allocator within each budget.
// Record of the corner widths (LD = 20) staged in LDS: the tile (0, 0) accumulators
// [lane][element], the summed strip of tile (0, 1) [lane column][element], the summed
// corner block [lane column][element], the right-hand side b[0..19], a zero for the
// padding entries, and a sink for the stores of lanes without an entry.
constexpr int kImgTile = 0, kImgStrip = 256, kImgCorner = 320, kImgRhs = 336, kImgZero = 356,
              kImgSink = 360, kImgFloats = 364;
constexpr int kRecordEntries20 = ne_floats(20);
static_assert(sizeof(GroupStage) >= sizeof(float) * kImgFloats, "the record image fits");
// Source in the image of every record entry (packed upper triangle of G, then b).
struct __attribute__((aligned(8))) RecordMap20 {
  uint16_t src[kRecordEntries20];
};
constexpr RecordMap20 make_record_map20() {
  RecordMap20 m{};
  constexpr int LD = 20, NTRI = LD * (LD + 1) / 2;
  for (int a = 0; a < LD; ++a) {
    for (int b = a; b < LD; ++b) {
      const int src = b < 16   ? kImgTile + 4 * (16 * (a >> 2) + b) + (a & 3)  // lane (a >> 2, b), element a & 3
                      : a < 16 ? kImgStrip + 4 * (4 * (a >> 2) + (b - 16)) + (a & 3)
                               : kImgCorner + 4 * (b - 16) + (a - 16);
      m.src[tri<LD>(a, b)] = (uint16_t)src;
    }
  }
  for (int d = 0; d < LD; ++d) m.src[NTRI + d] = (uint16_t)(kImgRhs + d);
  for (int e = NTRI + LD; e < kRecordEntries20; ++e) m.src[e] = (uint16_t)kImgZero;
  return m;
}
__constant__ RecordMap20 kRecordMap20 = make_record_map20();

template <int DP, int LD, bool AUG, bool WT, bool TS>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(TS ? 4 : WT ? 5 : 6)))
void k_gram_ne(const WorkItem *__restrict__ items, int64_t n_chunk_items,
               const int32_t *__restrict__ idx, const uint8_t *__restrict__ val,
               const float *__restrict__ wts, const float *__restrict__ Fp, int zrow,
               const float *__restrict__ Xold, int D, float *__restrict__ ws,
               float *__restrict__ ne, double *__restrict__ sse_out, Hadamard hd) {
  using C = RowCfg<DP>;
  constexpr int T = C::T, NT = C::NT;
  constexpr int NTRI = LD * (LD + 1) / 2;
  constexpr int NES = ne_floats(LD);
  static_assert(!AUG || (LD < DP && LD > 16 * (T - 1) && LD % 4 == 0),
                "the augmented column is feature LD of the last tile");
  // the last diagonal tile holds features 16 .. LD only: its 15 products go to VALU, and
  // the tile above it, which holds four used features, goes to 4 x 4 strips (STRIP)
  constexpr bool CORNER = AUG && T == 2 && LD == 20;
  constexpr bool STRIP = CORNER;
  __shared__ __attribute__((aligned(16))) GroupStage s_stage;
  const WorkItem it = items[blockIdx.x];
  const int lane = threadIdx.x, kq = lane >> 4, c = lane & 15;
  floatx4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  float rhs[T], xo[T];
#pragma unroll
  for (int X = 0; X < T; ++X) {
    rhs[X] = 0.f;
    {
      const float v = Xold[(int64_t)it.row * D + min(16 * X + c, D - 1)];
      xo[X] = 16 * X + c < D ? v : 0.f;
    }
  }
  double sse = 0.0;
  const float *__restrict__ wp = WT ? wts + it.start : nullptr;
  const int32_t *__restrict__ tp = TS ? hd.idx2 + it.start : nullptr;
  const GroupLanes g0 =
      first_group<WT, TS>(idx + it.start, val + it.start, wp, tp, it.len, zrow);
  // CORNER without the corner MFMA (TS): lane c < 15 of a row group owns the product
  // (cp, cq), cp <= cq < 5, of the features 16 + cp and 16 + cq (16 + 4 = LD is the
  // augmented column)
  int cp = 0, cq = 0;
  if constexpr (CORNER) {
    int rem = c;
    while (cp < 4 && rem >= 5 - cp) {
      rem -= 5 - cp;
      ++cp;
    }
    cq = c < 15 ? cp + rem : 0;
    if (c >= 15) cp = 0;
  }
  const int cx = (kq * 16 + cp) * 4, cy = (kq * 16 + cq) * 4;
  float corner = 0.f;
  gram_accumulate<DP, AUG, WT, TS, CORNER, STRIP>(acc, rhs, xo, sse, idx + it.start,
                                                  val + it.start, wp, tp, it.len, Fp, hd.Tp, zrow,
                                                  AUG ? LD - 16 * (T - 1) : -1, s_stage, g0,
                                                  corner, cx, cy);
  if constexpr (!AUG || STRIP) {
#pragma unroll
    for (int X = 0; X < T; ++X) {
      rhs[X] = sum_row_groups(rhs[X]);
    }
  }
  sse = sum_wave_f64(sse);
  float *__restrict__ out = ((int64_t)blockIdx.x < n_chunk_items ? ws : ne) + it.slot * NES;
  if constexpr (CORNER && !TS) {
    // The record is assembled in LDS (the staging area is free once the accumulation has
    // ended) with unmasked stores of each lane's values, then written with one coalesced
    // 16-byte store per lane, whose four entries come from the record map.
    static_assert(NES == kRecordEntries20 && LD == 20, "record map of the corner widths");
    float *const img = reinterpret_cast<float *>(&s_stage);
    *reinterpret_cast<floatx4 *>(img + kImgTile + 4 * lane) = acc[tidx<T>(0, 0)];
    floatx4 sv, cv;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      sv[r] = sum_row_groups(acc[tidx<T>(0, 1)][r]);
      cv[r] = sum_row_groups(acc[tidx<T>(1, 1)][r]);
    }
    corner = sum_row_groups(corner);
    // every row group holds the same sums: their stores to one address agree
    *reinterpret_cast<floatx4 *>(img + kImgStrip + 4 * c) = sv;
    *reinterpret_cast<floatx4 *>(c < 4 ? img + kImgCorner + 4 * c : img + kImgSink) = cv;
    img[kImgRhs + c] = rhs[0];
    img[c < 4 ? kImgRhs + 16 + c : kImgSink] = corner;
    img[kImgZero] = 0.f;
    wave_sync();
    if (lane < NES / 4) {
      const uint2 sp = *reinterpret_cast<const uint2 *>(&kRecordMap20.src[4 * lane]);
      const float4 o = make_float4(img[sp.x & 0xFFFF], img[sp.x >> 16], img[sp.y & 0xFFFF],
                                   img[sp.y >> 16]);
      *reinterpret_cast<float4 *>(out + 4 * lane) = o;
    }
    if (lane == 0) sse_out[blockIdx.x] = sse;
    return;
  }
  if constexpr (CORNER) {
    // (tensor ALS) lane c < 15 of a row group holds one corner product, summed over the
    // four rating groups
    corner = sum_row_groups(corner);
    if (kq == 0 && c < 15) {
      const int a = 16 + cp, b = 16 + cq;
      if (b < LD) out[tri<LD>(a, b)] = corner;
      else if (a < LD) out[NTRI + a] = corner;  // (a, LD): the right-hand side of feature a
    }
  }
  if constexpr (STRIP) {
    // the strip of tile (0, 1), summed over the four rating groups: lane c holds
    // G[4 (c >> 2) + r][16 + (c & 3)] in element r; the right-hand side of features 0..15
    // is rhs[0], summed above
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float v = acc[tidx<T>(0, 1)][r];
      v = sum_row_groups(v);
      if (kq == 0) out[tri<LD>(4 * (c >> 2) + r, 16 + (c & 3))] = v;
    }
    if (kq == 0) out[NTRI + c] = rhs[0];
  }
#pragma unroll
  for (int I = 0; I < T; ++I) {
#pragma unroll
    for (int J = I; J < T; ++J) {
      if (CORNER && I == T - 1) continue;
      if (STRIP && J == T - 1) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int a = 16 * I + 4 * kq + r, b = 16 * J + c;
        if (a <= b && b < LD) out[tri<LD>(a, b)] = acc[tidx<T>(I, J)][r];
        if constexpr (AUG) {
          // b_a = G[a][LD] sits in tile (I, T - 1), lane column LD - 16 (T - 1)
          if (J == T - 1 && b == LD && a < LD) out[NTRI + a] = acc[tidx<T>(I, J)][r];
        }
      }
    }
  }
  if constexpr (!AUG) {
    if (kq == 0) {
#pragma unroll
      for (int X = 0; X < T; ++X)
        if (16 * X + c < LD) out[NTRI + 16 * X + c] = rhs[X];
    }
  }
  if (lane == 0) sse_out[blockIdx.x] = sse;
}

// Sum the chunk records of each split row, in slot order, into the row's record.
template <int LD>
__global__ __launch_bounds__(256) void k_sum_records(const RowTask *__restrict__ rows, int64_t base,
                                                     const float *__restrict__ ws,
                                                     float *__restrict__ ne) {
  constexpr int NES = ne_floats(LD);
  const RowTask rt = rows[blockIdx.x];
  for (int e = threadIdx.x; e < NES; e += 256) {
    // unrolled so that several slots' loads are in flight before their additions, which
    // stay in slot order
    float v = 0.f;
#pragma unroll 8
    for (int s = 0; s < rt.nslots; ++s) v += ws[(rt.slot0 + s) * (int64_t)NES + e];
    ne[(base + blockIdx.x) * (int64_t)NES + e] = v;
  }
}

template <int LD, bool BAYES>
__global__ __launch_bounds__(64) void k_solve_lane(const RowTask *__restrict__ rows, int64_t n_rows,
                                                   int64_t base, const float *__restrict__ ne,
                                                   int D, float lam, float *__restrict__ X,
                                                   int32_t *__restrict__ flag_count,
                                                   RowPrior pr) {
  constexpr int NTRI = LD * (LD + 1) / 2;
  constexpr int NES = ne_floats(LD);
  constexpr int NQ = NES / 4;               // float4 of a record
  constexpr int ROUNDS = 4;                 // the records are read in four slices
  constexpr int QS = (NQ + ROUNDS - 1) / ROUNDS;
  constexpr int STRIDE = QS | 1;            // odd LDS row stride (in float4)
  __shared__ float4 s_rec[64 * STRIDE];
  const int lane = threadIdx.x;
  const int64_t first = (int64_t)blockIdx.x * 64;
  const int64_t i = first + lane;
  const int64_t nrec = n_rows - first < 64 ? n_rows - first : 64;  // >= 1
  const float4 *__restrict__ recs = reinterpret_cast<const float4 *>(ne) + (base + first) * NQ;
  float A[NTRI], b[LD];
  // The block's 64 records are contiguous: each slice is read with consecutive lanes on
  // consecutive float4 (record rr, float4 q0 + pc), staged in LDS, and every lane takes its
  // own record's part; lanes past the last row read the last record again.
#pragma unroll
  for (int h = 0; h < ROUNDS; ++h) {
    const int q0 = h * QS;
    const int nq = NQ - q0 < QS ? NQ - q0 : QS;
#pragma unroll
    for (int k = 0; k < QS; ++k) {
      if (k < nq) {
        const int f = k * 64 + lane;
        const int rr = f / nq, pc = f - rr * nq;
        const int64_t rec = rr < nrec ? rr : nrec - 1;
        s_rec[rr * STRIDE + pc] = recs[rec * NQ + q0 + pc];
      }
    }
    wave_sync();
#pragma unroll
    for (int pc = 0; pc < QS; ++pc) {
      if (pc < nq) {
        const float4 v = s_rec[lane * STRIDE + pc];
        const float w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int e = 4 * (q0 + pc) + j;
          if (e < NTRI) A[e] = w[j];
          else if (e < NTRI + LD) b[e - NTRI] = w[j];
        }
      }
    }
    wave_sync();  // the stage is refilled by the next slice
  }
  if (i >= n_rows) return;
  const RowTask rt = rows[i];
  if constexpr (BAYES) {
    // the prior image carries the identity on the padding; the time chain scales it per
    // row and adds the row's own right-hand side
    const float cs = pr.scale_of(rt.row);
#pragma unroll
    for (int e = 0; e < NTRI; ++e) A[e] = fmaf(cs, pr.init[e], A[e]);
#pragma unroll
    for (int d = 0; d < LD; ++d) b[d] = fmaf(cs, pr.init[NTRI + d], b[d]);
    if (pr.h0 != nullptr) {
      const float *__restrict__ hr = pr.h0 + (int64_t)rt.row * D;
#pragma unroll
      for (int d = 0; d < LD; ++d)
        if (d < D) b[d] += hr[d];
    }
  } else {
    const float lam_n = (float)((double)lam * (double)rt.deg);
#pragma unroll
    for (int d = 0; d < LD; ++d) A[tri<LD>(d, d)] = d < D ? A[tri<LD>(d, d)] + lam_n : 1.f;
  }

  // A = U^T U in place (upper triangle); the diagonal keeps 1 / u_kk
  bool bad = false;
#pragma unroll
  for (int k = 0; k < LD; ++k) {
    const float p = A[tri<LD>(k, k)];
    bad |= !(p > 0.f && p < INFINITY);
    const float iv = inv_sqrt_pivot(p);
    A[tri<LD>(k, k)] = iv;
#pragma unroll
    for (int j = k + 1; j < LD; ++j) A[tri<LD>(k, j)] *= iv;
#pragma unroll
    for (int r = k + 1; r < LD; ++r) {
#pragma unroll
      for (int j = r; j < LD; ++j)
        A[tri<LD>(r, j)] = fmaf(-A[tri<LD>(k, r)], A[tri<LD>(k, j)], A[tri<LD>(r, j)]);
    }
  }
  // U^T y = b (y overwrites b)
#pragma unroll
  for (int k = 0; k < LD; ++k) {
    b[k] *= A[tri<LD>(k, k)];
#pragma unroll
    for (int j = k + 1; j < LD; ++j) b[j] = fmaf(-A[tri<LD>(k, j)], b[k], b[j]);
  }
  if constexpr (BAYES) {
    const float *__restrict__ zr = pr.z + (int64_t)rt.row * D;
#pragma unroll
    for (int d = 0; d < LD; ++d)
      if (d < D) b[d] = fmaf(pr.zscale, zr[d], b[d]);
  }
  // U x = y (x overwrites b)
#pragma unroll
  for (int k = LD - 1; k >= 0; --k) {
    float s = b[k];
#pragma unroll
    for (int j = k + 1; j < LD; ++j) s = fmaf(-A[tri<LD>(k, j)], b[j], s);
    b[k] = s * A[tri<LD>(k, k)];
  }
#pragma unroll
  for (int d = 0; d < LD; ++d) bad |= !(fabsf(b[d]) < INFINITY);
  if (bad) {
    atomicAdd(flag_count, 1);
    return;
  }
  float *__restrict__ xr = X + (int64_t)rt.row * D;
#pragma unroll
  for (int d = 0; d < LD; ++d)
    if (d < D) xr[d] = b[d];
}

template <int DP, int LD, bool AUG>
static hipError_t launch_gram_ne_t(const WorkItem *items, int64_t n_items, int64_t n_chunk_items,
                                   const int32_t *idx, const uint8_t *val, const float *wts,
                                   const float *Fp, int zrow, const float *Xold, int D, float *ws,
                                   float *ne, double *sse, const Hadamard &hd, hipStream_t s) {
  if (hd.idx2) {
    // tensor ALS has no per-rating weights
    if (wts) return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_gram_ne<DP, LD, AUG, false, true>), dim3((unsigned)n_items), dim3(64),
                       0, s, items, n_chunk_items, idx, val, wts, Fp, zrow, Xold, D, ws, ne, sse,
                       hd);
  } else if (wts)
    hipLaunchKernelGGL((k_gram_ne<DP, LD, AUG, true, false>), dim3((unsigned)n_items), dim3(64),
                       0, s, items, n_chunk_items, idx, val, wts, Fp, zrow, Xold, D, ws, ne, sse,
                       hd);
  else
    hipLaunchKernelGGL((k_gram_ne<DP, LD, AUG, false, false>), dim3((unsigned)n_items), dim3(64),
                       0, s, items, n_chunk_items, idx, val, wts, Fp, zrow, Xold, D, ws, ne, sse,
                       hd);
  return hipSuccess;
}

hipError_t launch_gram_ne(int D, const WorkItem *items, int64_t n_items, int64_t n_chunk_items,
                          const int32_t *idx, const uint8_t *val, const float *wts,
                          const float *Fp, int64_t n_fixed, const float *Xold, float *ws,
                          float *ne, double *sse, const Hadamard &hd, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  const int zrow = (int)n_fixed;
  const int ld = lane_width(D);
  hipError_t e;
  if (ld == 16)
    e = launch_gram_ne_t<16, 16, false>(items, n_items, n_chunk_items, idx, val, wts, Fp, zrow,
                                        Xold, D, ws, ne, sse, hd, s);
  else if (ld == 20)
    e = launch_gram_ne_t<32, 20, true>(items, n_items, n_chunk_items, idx, val, wts, Fp, zrow,
                                       Xold, D, ws, ne, sse, hd, s);
  else
    return hipErrorInvalidValue;
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

template <int LD>
static void launch_solve_lane_t(unsigned blocks, const RowTask *rows, int64_t n_rows, int64_t base,
                                const float *ne, int D, float lam, float *X, int32_t *flag,
                                const RowPrior &pr, hipStream_t s) {
  if (pr.init)
    hipLaunchKernelGGL((k_solve_lane<LD, true>), dim3(blocks), dim3(64), 0, s, rows, n_rows, base,
                       ne, D, lam, X, flag, pr);
  else
    hipLaunchKernelGGL((k_solve_lane<LD, false>), dim3(blocks), dim3(64), 0, s, rows, n_rows,
                       base, ne, D, lam, X, flag, pr);
}

hipError_t launch_solve_lane(int D, const RowTask *rows, int64_t n_rows, int64_t n_split,
                             int64_t base, const float *ws, float *ne, float lam, float *X,
                             int32_t *flag, const RowPrior &pr, hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  const int ld = lane_width(D);
  if (ld != 16 && ld != 20) return hipErrorInvalidValue;
  if (n_split > 0) {
    if (ld == 16)
      hipLaunchKernelGGL(k_sum_records<16>, dim3((unsigned)n_split), dim3(256), 0, s, rows, base,
                         ws, ne);
    else
      hipLaunchKernelGGL(k_sum_records<20>, dim3((unsigned)n_split), dim3(256), 0, s, rows, base,
                         ws, ne);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const unsigned blocks = (unsigned)((n_rows + 63) / 64);
  if (ld == 16)
    launch_solve_lane_t<16>(blocks, rows, n_rows, base, ne, D, lam, X, flag, pr, s);
  else
    launch_solve_lane_t<20>(blocks, rows, n_rows, base, ne, D, lam, X, flag, pr, s);
  return hipGetLastError();
}

}  // namespace als
