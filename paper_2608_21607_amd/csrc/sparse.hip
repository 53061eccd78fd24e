// Sparse correction of the fused contraction at the nonzeros of S.
//
// The dense kernel contracts min(0, L) over every (i, j) of a block.  On the nonzeros of S the
// auxiliary matrix is S itself (eq. updateZ), so each nonzero adds (s_ij - min(0, l_ij)) p_j to
// row i of Y.  Work is split into items of at most a few hundred entries of one row (long rows
// are cut into several items whose partial results are summed afterwards in a fixed order), so
// power-law and Zipf rows do not serialise on one wavefront and the result is deterministic.
//
// A team of T lanes owns one item and keeps four of its entries in flight; lane t holds E = RP/T
// columns of the row's factor x_i and of its partial result: the E consecutive columns from
// t E when E is a multiple of 4 (16-byte accesses; 9% faster than the strided form on the graph
// workload), else columns t, t + T, ...  Either way a gather of a row p_j is one coalesced run
// of RP floats.  l_ij = x_i . p_j is reduced across the team with lane shuffles.  An item's
// terms and the fix-up's partial results are summed in fp64: on nearly full rows the fp32 sums
// of hundreds of terms, amplified by an ill-conditioned Gram matrix, had put W 2e-4 from the
// fp64 oracle after one sweep (7e-5 with fp64 sums; 7% more time for this kernel).

#include "nmd_internal.h"

namespace nmd {

// Column c of a row is held by lane c / E, element c % E when CONTIG (E consecutive floats per
// lane: one 16-byte access per four of them), else by lane c % T, element c / T.
template <int T, int E, bool CONTIG>
__device__ __forceinline__ int64_t col_of(int t, int e) {
  return CONTIG ? (int64_t)t * E + e : (int64_t)t + (int64_t)T * e;
}

template <int T, int E, bool CONTIG>
__device__ __forceinline__ void load_row(float (&v)[E], const float* __restrict__ src, int t) {
  if constexpr (CONTIG && E % 4 == 0) {
#pragma unroll
    for (int e = 0; e < E; e += 4) {
      const float4 w = *reinterpret_cast<const float4*>(src + (int64_t)t * E + e);
      v[e] = w.x;
      v[e + 1] = w.y;
      v[e + 2] = w.z;
      v[e + 3] = w.w;
    }
  } else {
#pragma unroll
    for (int e = 0; e < E; ++e) v[e] = src[col_of<T, E, CONTIG>(t, e)];
  }
}

template <int T, int E, bool CONTIG>
__device__ __forceinline__ void store_row(float* __restrict__ dst, const float (&v)[E], int t,
                                          bool add) {
  if constexpr (CONTIG && E % 4 == 0) {
#pragma unroll
    for (int e = 0; e < E; e += 4) {
      float4* d = reinterpret_cast<float4*>(dst + (int64_t)t * E + e);
      float4 w = make_float4(v[e], v[e + 1], v[e + 2], v[e + 3]);
      if (add) {
        const float4 o = *d;
        w.x += o.x;
        w.y += o.y;
        w.z += o.z;
        w.w += o.w;
      }
      *d = w;
    }
  } else {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      float* d = dst + col_of<T, E, CONTIG>(t, e);
      *d = add ? *d + v[e] : v[e];
    }
  }
}

template <int T, int E, int U, bool CONTIG>
__global__ __launch_bounds__(256) void sparse_kernel(const Item* __restrict__ items, int64_t nitems,
                                                     const int32_t* __restrict__ idx,
                                                     const float* __restrict__ val,
                                                     const float* __restrict__ X,
                                                     const float* __restrict__ P,
                                                     float* __restrict__ Y,
                                                     float* __restrict__ scratch,
                                                     int accumulate) {
  constexpr int RP = T * E;
  int64_t team = ((int64_t)blockIdx.x * 256 + threadIdx.x) / T;
  // a 64-lane team is one wave: its item index is uniform, so the item and its first entries
  // come through the scalar cache
  if constexpr (T == 64) team = (int64_t)__builtin_amdgcn_readfirstlane((int)team);
  const int t = threadIdx.x % T;
  if (team >= nitems) return;
  const Item it = items[team];
  const int64_t b = it.begin;
  const int cnt = it.count;
  // Everything that depends only on the item is requested at once: the factor row, the output
  // row it adds to, and the first U entries.  The gathers then wait for a single round trip.
  const bool rmw = it.slot < 0 && accumulate;
  float* const yrow = it.slot < 0 ? Y + (int64_t)it.row * RP : scratch + (int64_t)it.slot * RP;
  float x[E], yv[E];
  double acc[E];  // a row's terms are summed in fp64 (long rows have hundreds)
  load_row<T, E, CONTIG>(x, X + (int64_t)it.row * RP, t);
  if (rmw) load_row<T, E, CONTIG>(yv, yrow, t);
  int32_t jn[U];
  float sn[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const bool in = u < cnt;
    jn[u] = in ? idx[b + u] : 0;
    sn[u] = in ? val[b + u] : 0.f;
  }
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.0;
  int p = 0;
  for (; p + U <= cnt; p += U) {
    int32_t j[U];
    float s[U], pv[U][E], d[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      j[u] = jn[u];
      s[u] = sn[u];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) load_row<T, E, CONTIG>(pv[u], P + (int64_t)j[u] * RP, t);
    // the next group's entries, in flight during this group's arithmetic
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool in = p + U + u < cnt;
      jn[u] = in ? idx[b + p + U + u] : 0;
      sn[u] = in ? val[b + p + U + u] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float dd = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) dd = fmaf(x[e], pv[u][e], dd);
      d[u] = dd;
    }
#pragma unroll
    for (int off = T / 2; off > 0; off >>= 1)
#pragma unroll
      for (int u = 0; u < U; ++u) d[u] += __shfl_xor(d[u], off, T);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float c = s[u] - fminf(d[u], 0.f);
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] = fma((double)c, (double)pv[u][e], acc[e]);
    }
  }
  // the last cnt - p (< U) entries are in jn / sn: their rows are requested together before
  // any is used (one round trip, not one per entry); a slot past the end holds zeros and
  // adds nothing
  if (p < cnt) {
    float pv[U - 1][E], d[U - 1];
#pragma unroll
    for (int u = 0; u < U - 1; ++u) {
      if (p + u < cnt) {
        load_row<T, E, CONTIG>(pv[u], P + (int64_t)jn[u] * RP, t);
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) pv[u][e] = 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < U - 1; ++u) {
      float dd = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) dd = fmaf(x[e], pv[u][e], dd);
      d[u] = dd;
    }
#pragma unroll
    for (int off = T / 2; off > 0; off >>= 1)
#pragma unroll
      for (int u = 0; u < U - 1; ++u) d[u] += __shfl_xor(d[u], off, T);
#pragma unroll
    for (int u = 0; u < U - 1; ++u) {
      if (p + u < cnt) {
        const float c = sn[u] - fminf(d[u], 0.f);
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = fma((double)c, (double)pv[u][e], acc[e]);
      }
    }
  }
  if (rmw) {
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] += (double)yv[e];
  }
  float out[E];
#pragma unroll
  for (int e = 0; e < E; ++e) out[e] = (float)acc[e];
  store_row<T, E, CONTIG>(yrow, out, t, false);
}

template <int T, int E, bool CONTIG>
__global__ __launch_bounds__(256) void fixup_kernel(const Split* __restrict__ splits, int64_t n,
                                                    const float* __restrict__ scratch,
                                                    float* __restrict__ Y, int accumulate) {
  constexpr int RP = T * E;
  const int64_t team = ((int64_t)blockIdx.x * 256 + threadIdx.x) / T;
  const int t = threadIdx.x % T;
  if (team >= n) return;
  const Split sp = splits[team];
  double acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.0;
  for (int k = 0; k < sp.nslots; ++k) {
    float v[E];
    load_row<T, E, CONTIG>(v, scratch + (int64_t)(sp.first + k) * RP, t);
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] += (double)v[e];
  }
  float out[E];
#pragma unroll
  for (int e = 0; e < E; ++e) out[e] = (float)acc[e];
  store_row<T, E, CONTIG>(Y + (int64_t)sp.row * RP, out, t, accumulate != 0);
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

constexpr int kDepth = 4;  // entries of an item in flight per team (8: no faster)
constexpr bool contig(int E) { return E % 4 == 0; }

static inline unsigned grid_for(int64_t teams, int T) {
  return (unsigned)((teams * T + 255) / 256);
}

hipError_t launch_sparse(const Item* items, int64_t nitems, const int32_t* idx, const float* val,
                         const float* X, const float* P, int rp, float* Y, float* scratch,
                         int accumulate, hipStream_t st) {
  if (nitems <= 0) return hipSuccess;
#define LAUNCH(T, E)                                                                          \
  hipLaunchKernelGGL((sparse_kernel<T, E, kDepth, contig(E)>), dim3(grid_for(nitems, T)),      \
                     dim3(256), 0, st, items, nitems, idx, val, X, P, Y, scratch, accumulate)
  NMD_SPARSE_DISPATCH(rp, LAUNCH)
#undef LAUNCH
}

hipError_t launch_fixup(const Split* splits, int64_t nsplits, const float* scratch, int rp,
                        float* Y, int accumulate, hipStream_t st) {
  if (nsplits <= 0) return hipSuccess;
#define LAUNCH(T, E)                                                                           \
  hipLaunchKernelGGL((fixup_kernel<T, E, contig(E)>), dim3(grid_for(nsplits, T)), dim3(256), 0,  \
                     st, splits, nsplits, scratch, Y, accumulate)
  NMD_SPARSE_DISPATCH(rp, LAUNCH)
#undef LAUNCH
}

}  // namespace nmd
