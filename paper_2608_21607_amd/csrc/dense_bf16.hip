// Launchers of the rectified contraction with both products on split bf16 MFMA: the 32 x 32 x 16
// form at padded ranks 16 to 128 (kernels in dense_bf16.h), the 16 x 16 x 32 form at 256 and
// 512 (dense_bf16_large.hip).

#include "dense_bf16.h"
#include "nmd_internal.h"

namespace nmd {

bool bf16x3_rank(int rp) {
  return rp == 16 || rp == 32 || rp == 64 || rp == 128 || rp == 256 || rp == 512;
}

int64_t bf16x3_work_floats(int64_t blk, int rp) {
  if (rp >= 256) return blk * rp;  // the row-major copy only (read transposed in LDS)
  return blk * rp + (blk + 31) / 32 * 32 * (rp < 32 ? 32 : rp);
}

hipError_t launch_bf16x3(const float* X, int64_t rows, const float* P, int64_t blk, int rp,
                         float* work, float* Ypart, int64_t y_stride, int nsplit, float sgn,
                         unsigned long long* live, hipStream_t st) {
#define BX32(R) bx32_launch_t<R>(X, rows, P, blk, work, Ypart, y_stride, nsplit, sgn, live, st)
  switch (rp) {
    case 16: return BX32(16);
    case 32: return BX32(32);
    case 64: return BX32(64);
    case 128: return BX32(128);
    case 256:
    case 512:
      return launch_bf16x3_staged(X, rows, P, blk, rp, work, Ypart, y_stride, nsplit, sgn, live,
                                  st);
  }
#undef BX32
  return hipErrorInvalidValue;
}

int64_t bf16x3_pair_start(int s, int nsplit, int64_t blk) { return bx::pair_start(s, nsplit, blk); }

}  // namespace nmd
