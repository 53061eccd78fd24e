// The split-bf16 rectified contraction with its workspace in a static device array, for callers
// that cannot allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid hipMalloc).
//
// `scratch` holds the split copies of the panel that nmd_rectified_contraction_bf16x3 otherwise
// takes from a caller-owned workspace.  Each GPU the library runs on holds its own copy of the
// array until the process ends.  In host code the name `scratch` is not a device address: the
// address is looked up once per device with hipGetSymbolAddress (with that device current) and
// kept in g_ptr; only that pointer is ever passed to a kernel.

#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/nmd.h"
#include "nmd_internal.h"

namespace {

constexpr int64_t kScratchFloats = int64_t(4) << 20;  // 16 MiB per device
constexpr int kMaxDevices = 64;

static __device__ __align__(256) float scratch[kScratchFloats];

std::mutex g_mu;
float* g_ptr[kMaxDevices] = {};

}  // namespace

extern "C" int nmd_rectified_contraction_bf16x3_noalloc(const float* A, int64_t rows,
                                                       const float* B, int64_t blk, int32_t r,
                                                       float* Y, void* hip_stream) {
  if (!A || !B || !Y) return nmd::set_static_error(NMD_EINVAL, "A, B and Y must be non-NULL");
  if (rows < 1 || blk < 1 || rows > INT32_MAX)
    return nmd::set_static_error(NMD_EINVAL, "rows and blk must be >= 1");
  if (!nmd::bf16x3_rank(r))
    return nmd::set_static_error(
        NMD_EINVAL, "the bf16x3 contraction needs r in {16, 32, 64, 128, 256, 512} (got %d)", r);
  const int64_t need = nmd::bf16x3_work_floats(blk, r);
  if (need > kScratchFloats)
    return nmd::set_static_error(
        NMD_EINVAL,
        "a %lld-row panel at r = %d needs %lld floats of workspace; the static workspace holds "
        "%lld (use nmd_rectified_contraction_bf16x3 with a workspace of its own)",
        (long long)blk, r, (long long)need, (long long)kScratchFloats);
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess)
    return nmd::set_static_error(NMD_EDEVICE, "hipGetDevice failed: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return nmd::set_static_error(NMD_EDEVICE, "device %d is beyond the %d this entry point serves",
                                 dev, kMaxDevices);
  float* ws = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_ptr[dev]) {
      void* p = nullptr;
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return nmd::set_static_error(NMD_EDEVICE, "hipGetSymbolAddress of the workspace failed: %s",
                                     hipGetErrorString(e));
      g_ptr[dev] = static_cast<float*>(p);
    }
    ws = g_ptr[dev];
  }
  nmd::clear_static_error();
  e = nmd::launch_bf16x3(A, rows, B, blk, r, ws, Y, 0, 1, 1.0f, nullptr, (hipStream_t)hip_stream);
  if (e != hipSuccess)
    return nmd::set_static_error(NMD_EDEVICE, "launch failed: %s", hipGetErrorString(e));
  return NMD_OK;
}
