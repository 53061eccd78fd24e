// Sparse correction of the fused contraction at the nonzeros of S.
//
// The dense kernel contracts min(0, L) over every (i, j) of a block.  On the nonzeros of S the
// auxiliary matrix is S itself (eq. updateZ), so each nonzero adds (s_ij - min(0, l_ij)) p_j to
// row i of Y.  Work is split into items of at most a few hundred entries of one row (long rows
// are cut into several items whose partial results are summed afterwards in a fixed order), so
// power-law and Zipf rows do not serialise on one wavefront and the result is deterministic.
//
// A team of T lanes owns one item; lane t holds the E = RP/T columns t, t+T, ... of the row's
// factor x_i and of its partial result, so every gather of a row p_j is a coalesced run of RP
// floats.  l_ij = x_i . p_j is reduced across the team with lane shuffles.

#include "nmd_internal.h"

namespace nmd {

template <int T, int E>
__global__ __launch_bounds__(256) void sparse_kernel(const Item* __restrict__ items, int64_t nitems,
                                                     const int32_t* __restrict__ idx,
                                                     const float* __restrict__ val,
                                                     const float* __restrict__ X,
                                                     const float* __restrict__ P,
                                                     float* __restrict__ Y,
                                                     float* __restrict__ scratch,
                                                     int accumulate) {
  constexpr int RP = T * E;
  const int64_t team = ((int64_t)blockIdx.x * 256 + threadIdx.x) / T;
  const int t = threadIdx.x % T;
  if (team >= nitems) return;
  const Item it = items[team];
  const float* xr = X + (int64_t)it.row * RP;
  float x[E], acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    x[e] = xr[t + T * e];
    acc[e] = 0.f;
  }
  const int64_t b = it.begin;
  const int cnt = it.count;
  int p = 0;
  for (; p + 4 <= cnt; p += 4) {
    int32_t j[4];
    float s[4], pv[4][E], d[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      j[u] = idx[b + p + u];
      s[u] = val[b + p + u];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int e = 0; e < E; ++e) pv[u][e] = P[(int64_t)j[u] * RP + t + T * e];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      float dd = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) dd = fmaf(x[e], pv[u][e], dd);
      d[u] = dd;
    }
#pragma unroll
    for (int off = T / 2; off > 0; off >>= 1)
#pragma unroll
      for (int u = 0; u < 4; ++u) d[u] += __shfl_xor(d[u], off, T);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float c = s[u] - fminf(d[u], 0.f);
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] = fmaf(c, pv[u][e], acc[e]);
    }
  }
  for (; p < cnt; ++p) {
    const int32_t j = idx[b + p];
    const float s = val[b + p];
    float pv[E];
    float dd = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      pv[e] = P[(int64_t)j * RP + t + T * e];
      dd = fmaf(x[e], pv[e], dd);
    }
#pragma unroll
    for (int off = T / 2; off > 0; off >>= 1) dd += __shfl_xor(dd, off, T);
    const float c = s - fminf(dd, 0.f);
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = fmaf(c, pv[e], acc[e]);
  }
  if (it.slot < 0) {
    float* yr = Y + (int64_t)it.row * RP;
#pragma unroll
    for (int e = 0; e < E; ++e) yr[t + T * e] = accumulate ? yr[t + T * e] + acc[e] : acc[e];
  } else {
    float* sr = scratch + (int64_t)it.slot * RP;
#pragma unroll
    for (int e = 0; e < E; ++e) sr[t + T * e] = acc[e];
  }
}

template <int T, int E>
__global__ __launch_bounds__(256) void fixup_kernel(const Split* __restrict__ splits, int64_t n,
                                                    const float* __restrict__ scratch,
                                                    float* __restrict__ Y, int accumulate) {
  constexpr int RP = T * E;
  const int64_t team = ((int64_t)blockIdx.x * 256 + threadIdx.x) / T;
  const int t = threadIdx.x % T;
  if (team >= n) return;
  const Split sp = splits[team];
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  for (int k = 0; k < sp.nslots; ++k) {
    const float* sr = scratch + (int64_t)(sp.first + k) * RP;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] += sr[t + T * e];
  }
  float* yr = Y + (int64_t)sp.row * RP;
#pragma unroll
  for (int e = 0; e < E; ++e) yr[t + T * e] = accumulate ? yr[t + T * e] + acc[e] : acc[e];
}

#define NMD_SPARSE_DISPATCH(rp, LAUNCH) \
  switch (rp) {                         \
    case 16: LAUNCH(16, 1); break;      \
    case 32: LAUNCH(16, 2); break;      \
    case 48: LAUNCH(16, 3); break;      \
    case 64: LAUNCH(16, 4); break;      \
    case 128: LAUNCH(64, 2); break;     \
    case 192: LAUNCH(64, 3); break;     \
    case 256: LAUNCH(64, 4); break;     \
    case 320: LAUNCH(64, 5); break;     \
    case 384: LAUNCH(64, 6); break;     \
    case 448: LAUNCH(64, 7); break;     \
    case 512: LAUNCH(64, 8); break;     \
    default: return hipErrorInvalidValue; \
  }                                     \
  return hipGetLastError();

static inline unsigned grid_for(int64_t teams, int T) {
  return (unsigned)((teams * T + 255) / 256);
}

hipError_t launch_sparse(const Item* items, int64_t nitems, const int32_t* idx, const float* val,
                         const float* X, const float* P, int rp, float* Y, float* scratch,
                         int accumulate, hipStream_t st) {
  if (nitems <= 0) return hipSuccess;
#define LAUNCH(T, E)                                                                          \
  hipLaunchKernelGGL((sparse_kernel<T, E>), dim3(grid_for(nitems, T)), dim3(256), 0, st, items, \
                     nitems, idx, val, X, P, Y, scratch, accumulate)
  NMD_SPARSE_DISPATCH(rp, LAUNCH)
#undef LAUNCH
}

hipError_t launch_fixup(const Split* splits, int64_t nsplits, const float* scratch, int rp,
                        float* Y, int accumulate, hipStream_t st) {
  if (nsplits <= 0) return hipSuccess;
#define LAUNCH(T, E)                                                                           \
  hipLaunchKernelGGL((fixup_kernel<T, E>), dim3(grid_for(nsplits, T)), dim3(256), 0, st, splits, \
                     nsplits, scratch, Y, accumulate)
  NMD_SPARSE_DISPATCH(rp, LAUNCH)
#undef LAUNCH
}

}  // namespace nmd
