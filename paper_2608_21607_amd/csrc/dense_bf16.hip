// Launchers of the rectified contraction with both products on split bf16 MFMA (kernels in
// dense_bf16.h): the 32 x 32 x 16 form at padded ranks 32, 64, 128, the 16 x 16 x 32 form at 256.

#include "dense_bf16.h"
#include "nmd_internal.h"

namespace nmd {

int64_t bf16x3_work_floats(int64_t blk, int rp) { return (blk + (blk + 31) / 32 * 32) * rp; }

template <int RP>
static hipError_t bx_launch_t(const float* X, int64_t rows, const float* P, int64_t blk,
                              float* work, float* Ypart, int64_t y_stride, int nsplit, float sgn,
                              unsigned long long* live, hipStream_t st) {
  using C = bx::Cfg<RP>;
  const int64_t npair = (blk + 31) / 32;
  float* rowm = work;
  float* trans = work + blk * RP;
  const int64_t threads = blk * (RP / 8) + npair * 4 * RP;
  hipLaunchKernelGGL(bx::bx_split_kernel<RP>, dim3((unsigned)((threads + 255) / 256)), dim3(256),
                     0, st, P, blk, npair, reinterpret_cast<bx::u32x4*>(rowm),
                     reinterpret_cast<bx::u32x4*>(trans));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t row_tiles = (rows + C::ROWS - 1) / C::ROWS;
  const int64_t total = row_tiles * nsplit;
  if (total <= 0) return hipSuccess;
  if (total > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(bx::bx_kernel<RP>, dim3((unsigned)total), dim3(64 * C::WAVES), 0, st, X, rows,
                     rowm, trans, blk, Ypart, y_stride, nsplit, row_tiles, sgn, live);
  return hipGetLastError();
}

// Ranks up to 128: 32 rows of X per wave on the 32 x 32 x 16 MFMA.
template <int RP>
static hipError_t bx32_launch_t(const float* X, int64_t rows, const float* P, int64_t blk,
                                float* work, float* Ypart, int64_t y_stride, int nsplit,
                                float sgn, unsigned long long* live, hipStream_t st) {
  using C = bx::Cfg32<RP>;
  const int64_t npair = (blk + 31) / 32;
  float* rowm = work;
  float* trans = work + blk * RP;
  const int64_t threads = blk * (RP / 8) + npair * 4 * RP;
  hipLaunchKernelGGL(bx::bx32_split_kernel<RP>, dim3((unsigned)((threads + 255) / 256)),
                     dim3(256), 0, st, P, blk, npair, reinterpret_cast<bx::u32x4*>(rowm),
                     reinterpret_cast<bx::u32x4*>(trans));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t row_tiles = (rows + C::ROWS - 1) / C::ROWS;
  const int64_t total = row_tiles * nsplit;
  if (total <= 0) return hipSuccess;
  if (total > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(bx::bx32_kernel<RP>, dim3((unsigned)total), dim3(64 * C::WAVES), 0, st, X,
                     rows, rowm, trans, blk, Ypart, y_stride, nsplit, row_tiles, sgn, live);
  return hipGetLastError();
}

hipError_t launch_bf16x3(const float* X, int64_t rows, const float* P, int64_t blk, int rp,
                         float* work, float* Ypart, int64_t y_stride, int nsplit, float sgn,
                         unsigned long long* live, hipStream_t st) {
#define BX(R) bx_launch_t<R>(X, rows, P, blk, work, Ypart, y_stride, nsplit, sgn, live, st)
#define BX32(R) bx32_launch_t<R>(X, rows, P, blk, work, Ypart, y_stride, nsplit, sgn, live, st)
  switch (rp) {
    case 32: return BX32(32);
    case 64: return BX32(64);
    case 128: return BX32(128);
    case 256: return BX(256);
  }
#undef BX
#undef BX32
  return hipErrorInvalidValue;
}

int64_t bf16x3_pair_start(int s, int nsplit, int64_t blk) { return bx::pair_start(s, nsplit, blk); }

}  // namespace nmd
