// Launchers of the split-bf16 dense contraction at r_p = 256 (kernels in dense_split.h).

#include "dense_split.h"

namespace nmd {

hipError_t launch_split_panel(const float* P, int64_t rows, float* out, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  const int64_t threads = rows * 32;
  hipLaunchKernelGGL(split_panel_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0,
                     st, P, rows, reinterpret_cast<uintx4*>(out));
  return hipGetLastError();
}

hipError_t launch_dense_split(const float* X, int64_t rows, const float* Psplit, int64_t blk,
                              float* Ypart, int64_t y_stride, int nsplit, float sgn,
                              unsigned long long* gemm2_blocks, hipStream_t st) {
  const int64_t row_tiles = (rows + dense_rows<256>() - 1) / dense_rows<256>();
  const int64_t total = row_tiles * nsplit;
  if (total <= 0) return hipSuccess;
  if (total > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(dense_split_kernel, dim3((unsigned)total),
                     dim3(64 * DenseLaunch<256>::WAVES), 0, st, X, rows, Psplit, blk, Ypart,
                     y_stride, nsplit, row_tiles, sgn, gemm2_blocks);
  return hipGetLastError();
}

}  // namespace nmd
