// Kernel instantiations of the fused dense contraction for r_p >= 320 (one wave per SIMD).
// They are compiled with the MFMA accumulators in accumulation registers: with 512 registers
// per lane the output tiles live there and the ordinary VGPRs keep X, the operand ring and the
// panel fragments.

#include "dense_kernel.h"

namespace nmd {

hipError_t dense_wgs_per_cu_large(int rp, int* out) {
  switch (rp) {
    case 320: return wgs_per_cu_t<320>(out);
    case 384: return wgs_per_cu_t<384>(out);
    case 448: return wgs_per_cu_t<448>(out);
    case 512: return wgs_per_cu_t<512>(out);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_dense_large(const float* X, int64_t rows, const float* P, int64_t blk, int rp,
                              float* Ypart, int64_t y_stride, int nsplit, float sgn,
                              unsigned long long* gemm2_blocks, hipStream_t st) {
#define CALL(R) launch_dense_t<R>(X, rows, P, blk, Ypart, y_stride, nsplit, sgn, gemm2_blocks, st)
  switch (rp) {
    case 320: return CALL(320);
    case 384: return CALL(384);
    case 448: return CALL(448);
    case 512: return CALL(512);
  }
#undef CALL
  return hipErrorInvalidValue;
}

}  // namespace nmd
