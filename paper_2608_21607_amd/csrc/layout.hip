// Layout helpers: the caller's W (m x r) and H (r x n) <-> the padded panels A (m x rp) and
// B = H^T (n x rp) the kernels work on, plus a fill and an ordered fp64 reduction.

#include "nmd_internal.h"

namespace nmd {

__global__ void pad_rows_kernel(const float* __restrict__ src, int64_t rows, int r,
                                float* __restrict__ dst, int rp) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= rows * rp) return;
  const int64_t i = e / rp;
  const int c = (int)(e - i * rp);
  dst[e] = c < r ? src[i * r + c] : 0.f;
}

__global__ void unpad_rows_kernel(const float* __restrict__ src, int64_t rows, int rp,
                                  float* __restrict__ dst, int r) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= rows * r) return;
  const int64_t i = e / r;
  const int c = (int)(e - i * r);
  dst[e] = src[i * rp + c];
}

// 32 x 32 tiles through LDS: B[j][c] = H[c][j] (c < r), 0 for r <= c < rp.
__global__ void transpose_in_kernel(const float* __restrict__ H, int r, int64_t n,
                                    float* __restrict__ B, int rp) {
  __shared__ float t[32][33];
  const int64_t j0 = (int64_t)blockIdx.x * 32;
  const int c0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 256 threads: 32 x 8
  for (int k = ty; k < 32; k += 8) {
    const int c = c0 + k;
    const int64_t j = j0 + tx;
    t[k][tx] = (c < r && j < n) ? H[(int64_t)c * n + j] : 0.f;
  }
  __syncthreads();
  for (int k = ty; k < 32; k += 8) {
    const int64_t j = j0 + k;
    const int c = c0 + tx;
    if (j < n && c < rp) B[j * rp + c] = t[tx][k];
  }
}

__global__ void transpose_out_kernel(const float* __restrict__ B, int rp, int64_t n,
                                     float* __restrict__ H, int r) {
  __shared__ float t[32][33];
  const int64_t j0 = (int64_t)blockIdx.x * 32;
  const int c0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int k = ty; k < 32; k += 8) {
    const int64_t j = j0 + k;
    const int c = c0 + tx;
    t[k][tx] = (j < n && c < rp) ? B[j * rp + c] : 0.f;
  }
  __syncthreads();
  for (int k = ty; k < 32; k += 8) {
    const int c = c0 + k;
    const int64_t j = j0 + tx;
    if (c < r && j < n) H[(int64_t)c * n + j] = t[tx][k];
  }
}

__global__ void zero_kernel(float* __restrict__ p, int64_t count) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < count) p[e] = 0.f;
}

// A copy that does nothing once the status word holds a failure (the snapshot of the factors
// before a sweep must not be overwritten by the state after a sweep that was rejected).
__global__ void guarded_copy_kernel(const float4* __restrict__ src, float4* __restrict__ dst,
                                    int64_t n4, const int* status) {
  if (*(volatile const int*)status != 0) return;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < n4) dst[e] = src[e];
}

__global__ void guarded_copy_tail_kernel(const float* __restrict__ src, float* __restrict__ dst,
                                         int64_t begin, int64_t count, const int* status) {
  if (*(volatile const int*)status != 0) return;
  const int64_t e = begin + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e < count) dst[e] = src[e];
}

__global__ void guard_kernel(const double* __restrict__ q_old, const double* __restrict__ q_new,
                             double tol2, int* status, int step_id) {
  if (threadIdx.x != 0 || *(volatile const int*)status != 0) return;
  if (!(*q_new <= tol2 * *q_old)) {
    flag_status(status, STATUS_RISE, step_id);
  }
}

// One workgroup: per-thread strided partial sums, then a fixed-order tree.
__global__ __launch_bounds__(256) void sum_kernel(const double* __restrict__ partial,
                                                  int64_t count, double* __restrict__ out) {
  __shared__ double red[256];
  double s = 0.0;
  for (int64_t e = threadIdx.x; e < count; e += 256) s += partial[e];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int k = 128; k > 0; k >>= 1) {
    if ((int)threadIdx.x < k) red[threadIdx.x] += red[threadIdx.x + k];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = red[0];
}

static inline unsigned blocks(int64_t n) { return (unsigned)((n + 255) / 256); }

hipError_t launch_pad_rows(const float* src, int64_t rows, int r, float* dst, int rp,
                           hipStream_t st) {
  if (rows * rp == 0) return hipSuccess;
  hipLaunchKernelGGL(pad_rows_kernel, dim3(blocks(rows * rp)), dim3(256), 0, st, src, rows, r, dst, rp);
  return hipGetLastError();
}

hipError_t launch_unpad_rows(const float* src, int64_t rows, int rp, float* dst, int r,
                             hipStream_t st) {
  if (rows * r == 0) return hipSuccess;
  hipLaunchKernelGGL(unpad_rows_kernel, dim3(blocks(rows * r)), dim3(256), 0, st, src, rows, rp, dst, r);
  return hipGetLastError();
}

hipError_t launch_transpose_in(const float* H, int r, int64_t n, float* B, int rp,
                               hipStream_t st) {
  const dim3 grid((unsigned)((n + 31) / 32), (unsigned)((rp + 31) / 32));
  hipLaunchKernelGGL(transpose_in_kernel, grid, dim3(256), 0, st, H, r, n, B, rp);
  return hipGetLastError();
}

hipError_t launch_transpose_out(const float* B, int rp, int64_t n, float* H, int r,
                                hipStream_t st) {
  const dim3 grid((unsigned)((n + 31) / 32), (unsigned)((r + 31) / 32));
  hipLaunchKernelGGL(transpose_out_kernel, grid, dim3(256), 0, st, B, rp, n, H, r);
  return hipGetLastError();
}

hipError_t launch_zero(float* p, int64_t count, hipStream_t st) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_kernel, dim3(blocks(count)), dim3(256), 0, st, p, count);
  return hipGetLastError();
}

hipError_t launch_guarded_copy(const float* src, float* dst, int64_t count, const int* status,
                               hipStream_t st) {
  const int64_t n4 = count / 4;
  if (n4 > 0 && ((uintptr_t)src % 16 == 0) && ((uintptr_t)dst % 16 == 0)) {
    hipLaunchKernelGGL(guarded_copy_kernel, dim3(blocks(n4)), dim3(256), 0, st,
                       (const float4*)src, (float4*)dst, n4, status);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (count > 4 * n4)
      hipLaunchKernelGGL(guarded_copy_tail_kernel, dim3(1), dim3(256), 0, st, src, dst, 4 * n4,
                         count, status);
    return hipGetLastError();
  }
  if (count > 0)
    hipLaunchKernelGGL(guarded_copy_tail_kernel, dim3(blocks(count)), dim3(256), 0, st, src, dst,
                       (int64_t)0, count, status);
  return hipGetLastError();
}

hipError_t launch_guard(const double* q_old, const double* q_new, double tol2, int* status,
                        int step_id, hipStream_t st) {
  hipLaunchKernelGGL(guard_kernel, dim3(1), dim3(64), 0, st, q_old, q_new, tol2, status, step_id);
  return hipGetLastError();
}

hipError_t launch_sum(const double* partial, int64_t count, double* out, hipStream_t st) {
  hipLaunchKernelGGL(sum_kernel, dim3(1), dim3(256), 0, st, partial, count, out);
  return hipGetLastError();
}

}  // namespace nmd
