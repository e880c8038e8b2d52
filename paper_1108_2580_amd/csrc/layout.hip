// Device-side dual layout: the item-major (CSC) copy of the user-major CSR.
//
// The alternation of Sec. 2.2 needs both access directions: the user
// half-sweep walks each user's ratings, the item half-sweep each item's. The
// transpose is a stable counting sort done in four integer passes, so the
// result is bit-exact and reproducible (users ascend inside every column):
//
//  1. count:   rows are cut into blocks of R consecutive rows; cnt[b][c] counts
//              the ratings of column c inside row block b (integer atomics).
//  2. colscan: for each column, an exclusive prefix over the blocks turns cnt
//              into the block's starting offset inside the column, and the
//              column total is kept.
//  3. scan:    exclusive prefix over the column totals -> col_ptr.
//  4. scatter: one wavefront per row block walks its rows in order; within a
//              row the columns are distinct, so each rating claims the next
//              position of its column with an integer atomic; a fence between
//              rows keeps the claims of consecutive rows in row order.
#include "internal.h"

namespace als {

__global__ void k_fill_i32(int32_t *__restrict__ p, int64_t n, int32_t v) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = v;
}

hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_fill_i32, dim3((unsigned)blocks), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_csc_count(const int64_t *__restrict__ row_ptr,
                                                   const int32_t *__restrict__ col,
                                                   int64_t n_rows, int64_t n_cols,
                                                   int64_t rows_per_blk,
                                                   int32_t *__restrict__ cnt) {
  const int64_t b = blockIdx.x;
  const int64_t r0 = b * rows_per_blk;
  const int64_t r1 = r0 + rows_per_blk < n_rows ? r0 + rows_per_blk : n_rows;
  const int64_t p0 = row_ptr[r0], p1 = row_ptr[r1];
  int32_t *cb = cnt + b * n_cols;
  for (int64_t p = p0 + threadIdx.x; p < p1; p += blockDim.x) atomicAdd(&cb[col[p]], 1);
}

__global__ __launch_bounds__(256) void k_csc_colscan(int32_t *__restrict__ cnt, int64_t nblk,
                                                     int64_t n_cols, int64_t *__restrict__ tot) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= n_cols) return;
  int64_t run = 0;
  for (int64_t b = 0; b < nblk; ++b) {
    const int32_t v = cnt[b * n_cols + c];
    cnt[b * n_cols + c] = (int32_t)run;
    run += v;
  }
  tot[c] = run;
}

// Exclusive prefix sum of n int64 values into out[0..n] (out[n] = total), one
// workgroup of 1024 threads; thread t owns a contiguous range of inputs.
__global__ __launch_bounds__(1024) void k_scan_excl_i64(const int64_t *__restrict__ in, int64_t n,
                                                        int64_t *__restrict__ out) {
  __shared__ int64_t part[1024];
  const int t = threadIdx.x;
  const int64_t per = (n + 1023) / 1024;
  const int64_t b = t * per;
  const int64_t e = b + per < n ? b + per : n;
  int64_t s = 0;
  for (int64_t i = b; i < e; ++i) s += in[i];
  part[t] = s;
  __syncthreads();
  if (t == 0) {
    int64_t run = 0;
    for (int i = 0; i < 1024; ++i) {
      const int64_t v = part[i];
      part[i] = run;
      run += v;
    }
    out[n] = run;
  }
  __syncthreads();
  int64_t run = part[t];
  for (int64_t i = b; i < e; ++i) {
    out[i] = run;
    run += in[i];
  }
}

__global__ __launch_bounds__(64) void k_csc_scatter(const int64_t *__restrict__ row_ptr,
                                                    const int32_t *__restrict__ col,
                                                    const uint8_t *__restrict__ val,
                                                    int64_t n_rows, int64_t n_cols,
                                                    int64_t rows_per_blk, int32_t *cnt,
                                                    const int64_t *__restrict__ col_ptr,
                                                    int32_t *__restrict__ row_idx,
                                                    uint8_t *__restrict__ val_t) {
  const int64_t b = blockIdx.x;
  const int64_t r0 = b * rows_per_blk;
  const int64_t r1 = r0 + rows_per_blk < n_rows ? r0 + rows_per_blk : n_rows;
  int32_t *cb = cnt + b * n_cols;
  for (int64_t r = r0; r < r1; ++r) {
    const int64_t p1 = row_ptr[r + 1];
    for (int64_t p = row_ptr[r] + threadIdx.x; p < p1; p += 64) {
      const int32_t c = col[p];
      const int32_t k = atomicAdd(&cb[c], 1);
      const int64_t pos = col_ptr[c] + k;
      row_idx[pos] = (int32_t)r;
      val_t[pos] = val[p];
    }
    // claims of row r complete before any claim of row r + 1
    __threadfence();
  }
}

hipError_t launch_csc_build(const int64_t *row_ptr, const int32_t *col, const uint8_t *val,
                            int64_t n_rows, int64_t n_cols, int64_t rows_per_blk, int64_t nblk,
                            int32_t *scratch_cnt, int64_t *tot, int64_t *col_ptr,
                            int32_t *row_idx, uint8_t *val_t, hipStream_t s) {
  hipError_t e = launch_fill_i32(scratch_cnt, nblk * n_cols, 0, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_csc_count, dim3((unsigned)nblk), dim3(256), 0, s, row_ptr, col, n_rows,
                     n_cols, rows_per_blk, scratch_cnt);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_csc_colscan, dim3((unsigned)((n_cols + 255) / 256)), dim3(256), 0, s,
                     scratch_cnt, nblk, n_cols, tot);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_scan_excl_i64, dim3(1), dim3(1024), 0, s, tot, n_cols, col_ptr);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_csc_scatter, dim3((unsigned)nblk), dim3(64), 0, s, row_ptr, col, val,
                     n_rows, n_cols, rows_per_blk, scratch_cnt, col_ptr, row_idx, val_t);
  return hipGetLastError();
}

__global__ __launch_bounds__(64) void k_csc_scatter_f32(const int64_t *__restrict__ row_ptr,
                                                        const int32_t *__restrict__ col,
                                                        const float *__restrict__ w,
                                                        int64_t n_rows, int64_t n_cols,
                                                        int64_t rows_per_blk, int32_t *cnt,
                                                        const int64_t *__restrict__ col_ptr,
                                                        float *__restrict__ w_t) {
  const int64_t b = blockIdx.x;
  const int64_t r0 = b * rows_per_blk;
  const int64_t r1 = r0 + rows_per_blk < n_rows ? r0 + rows_per_blk : n_rows;
  int32_t *cb = cnt + b * n_cols;
  for (int64_t r = r0; r < r1; ++r) {
    const int64_t p1 = row_ptr[r + 1];
    for (int64_t p = row_ptr[r] + threadIdx.x; p < p1; p += 64) {
      const int32_t c = col[p];
      const int32_t k = atomicAdd(&cb[c], 1);
      w_t[col_ptr[c] + k] = w[p];
    }
    // claims of row r complete before any claim of row r + 1
    __threadfence();
  }
}

hipError_t launch_csc_permute_f32(const int64_t *row_ptr, const int32_t *col, const float *w,
                                  int64_t n_rows, int64_t n_cols, int64_t rows_per_blk,
                                  int64_t nblk, int32_t *scratch_cnt, int64_t *tot,
                                  const int64_t *col_ptr, float *w_t, hipStream_t s) {
  hipError_t e = launch_fill_i32(scratch_cnt, nblk * n_cols, 0, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_csc_count, dim3((unsigned)nblk), dim3(256), 0, s, row_ptr, col, n_rows,
                     n_cols, rows_per_blk, scratch_cnt);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_csc_colscan, dim3((unsigned)((n_cols + 255) / 256)), dim3(256), 0, s,
                     scratch_cnt, nblk, n_cols, tot);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(k_csc_scatter_f32, dim3((unsigned)nblk), dim3(64), 0, s, row_ptr, col, w,
                     n_rows, n_cols, rows_per_blk, scratch_cnt, col_ptr, w_t);
  return hipGetLastError();
}

// ---- fixed-order reduction of doubles --------------------------------------------------

constexpr int kRedBlock = 256;
constexpr int kRedPer = 8;  // values per thread per block

int64_t reduce_partials(int64_t n) {
  const int64_t per_blk = (int64_t)kRedBlock * kRedPer;
  return n > 0 ? (n + per_blk - 1) / per_blk : 1;
}

__device__ __forceinline__ double block_tree_sum(double v, double *sh) {
  sh[threadIdx.x] = v;
  __syncthreads();
  for (int w = kRedBlock / 2; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) sh[threadIdx.x] += sh[threadIdx.x + w];
    __syncthreads();
  }
  return sh[0];
}

// Block b sums v[b*2048 .. b*2048+2047]: thread t takes elements t, t+256, ...
// in order, then a fixed tree over the threads.
__global__ __launch_bounds__(kRedBlock) void k_reduce_partial(const double *__restrict__ v,
                                                              int64_t n,
                                                              double *__restrict__ partial) {
  __shared__ double sh[kRedBlock];
  const int64_t base = (int64_t)blockIdx.x * kRedBlock * kRedPer;
  double s = 0.0;
#pragma unroll
  for (int m = 0; m < kRedPer; ++m) {
    const int64_t i = base + threadIdx.x + (int64_t)m * kRedBlock;
    if (i < n) s += v[i];
  }
  const double tot = block_tree_sum(s, sh);
  if (threadIdx.x == 0) partial[blockIdx.x] = tot;
}

// One block: thread t sums partials t, t+256, ... in order, then a fixed tree. On request
// thread 0 also stores the total, and a copy of *flag, into mapped host memory, in place of
// two device-to-host copies after the kernel.
__global__ __launch_bounds__(kRedBlock) void k_reduce_final(const double *__restrict__ partial,
                                                            int64_t np, double *__restrict__ out,
                                                            double *host_out,
                                                            const int32_t *__restrict__ flag,
                                                            int32_t *host_flag) {
  __shared__ double sh[kRedBlock];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < np; i += kRedBlock) s += partial[i];
  const double tot = block_tree_sum(s, sh);
  if (threadIdx.x == 0) {
    *out = tot;
    if (host_out) *host_out = tot;
    if (host_flag) *host_flag = *flag;
  }
}

hipError_t launch_reduce(const double *v, int64_t n, double *partials, double *out,
                         hipStream_t s, double *host_out, const int32_t *flag,
                         int32_t *host_flag) {
  if ((flag == nullptr) != (host_flag == nullptr)) return hipErrorInvalidValue;
  const int64_t np = n > 0 ? reduce_partials(n) : 0;
  if (n > 0) {
    hipLaunchKernelGGL(k_reduce_partial, dim3((unsigned)np), dim3(kRedBlock), 0, s, v, n,
                       partials);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_reduce_final, dim3(1), dim3(kRedBlock), 0, s, partials, np, out, host_out,
                     flag, host_flag);
  return hipGetLastError();
}

}  // namespace als
