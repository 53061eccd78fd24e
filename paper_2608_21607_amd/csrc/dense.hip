// Fused dense contraction: launch shapes and dispatch for every padded rank, and the kernel
// instantiations for r_p <= 256 (compiled with MFMA accumulators in ordinary VGPRs).  The
// instantiations for r_p >= 320 are in dense_large.hip.

#include "dense_kernel.h"

namespace nmd {

int padded_rank(int r) {
  if (r <= 64) return ((r + 15) / 16) * 16;
  return ((r + 63) / 64) * 64;
}

int dense_max_wgs(int64_t rows, int rp, int nsplit) {
  const int rw = dense_rows_per_wg(rp);
  return rw ? (int)(((rows + rw - 1) / rw) * nsplit) : 0;
}

int dense_rows_per_wg(int rp) {
#define RW(R) dense_rows<R>()
  switch (rp) {
    case 16: return RW(16);
    case 32: return RW(32);
    case 48: return RW(48);
    case 64: return RW(64);
    case 128: return RW(128);
    case 192: return RW(192);
    case 256: return RW(256);
    case 320: return RW(320);
    case 384: return RW(384);
    case 448: return RW(448);
    case 512: return RW(512);
  }
#undef RW
  return 0;
}

hipError_t dense_wgs_per_cu(int rp, int* out) {
#define CALL(R) wgs_per_cu_t<R>(out)
  switch (rp) {
    case 16: return CALL(16);
    case 32: return CALL(32);
    case 48: return CALL(48);
    case 64: return CALL(64);
    case 128: return CALL(128);
    case 192: return CALL(192);
    case 256: return CALL(256);
    case 320: case 384: case 448: case 512: return dense_wgs_per_cu_large(rp, out);
  }
#undef CALL
  return hipErrorInvalidValue;
}

hipError_t launch_dense(const float* X, int64_t rows, const float* P, int64_t blk, int rp,
                        float* Ypart, int64_t y_stride, int nsplit, float sgn,
                        unsigned long long* gemm2_blocks, hipStream_t st) {
#define CALL(R) launch_dense_t<R>(X, rows, P, blk, Ypart, y_stride, nsplit, sgn, gemm2_blocks, st)
  switch (rp) {
    case 16: return CALL(16);
    case 32: return CALL(32);
    case 48: return CALL(48);
    case 64: return CALL(64);
    case 128: return CALL(128);
    case 192: return CALL(192);
    case 256: return CALL(256);
    case 320: case 384: case 448: case 512:
      return launch_dense_large(X, rows, P, blk, rp, Ypart, y_stride, nsplit, sgn, gemm2_blocks, st);
  }
#undef CALL
  return hipErrorInvalidValue;
}

}  // namespace nmd
