// Objective of eq. auxCost with Z eliminated (eq. SLloss):
//   f^2 ||S||_F^2 = sum_{S_ij = 0} max(0, L_ij)^2 + sum_{S_ij > 0} (S_ij - L_ij)^2,  L = X P^T,
// and, in the metrics variant, the reconstruction measures of S-hat = max(0, L) (eq. rectify):
//   RMSE (eq. RMSE)  E^2 ||S||_F^2 = sum_{S_ij = 0} S-hat_ij^2 + sum_{S_ij > 0} (S_ij - S-hat_ij)^2,
//   WJD  (eq. WJD)   J = 1 - sum min(S, S-hat) / sum max(S, S-hat).
// Off the nonzeros the three share max(0, L)^2 and max(0, L), so the kernel keeps five sums:
// q0 = sum_{S=0} max(0, L)^2, q1 = sum_{S>0} (S - L)^2, q2 = sum_{S>0} (S - S-hat)^2,
// q3 = sum_{S>0} min(S, S-hat), q4 = sum_{S=0} max(0, L) + sum_{S>0} max(S, S-hat).
//
// Every entry of L is formed once, on MFMA, exactly as in the fused contraction (same tiles,
// same transposed layout).  Each lane owns one row i and four columns 4q..4q+3 of every
// 16-column block, and walks row i's nonzeros of the current column block (sorted by column) in
// step with the tile loop; an entry that falls on one of its four columns switches that term
// from max(0, L)^2 to (S - L)^2.  So each term of eq. SLloss is taken once from the same L:
// nothing is added over all entries and subtracted again at the nonzeros (which would cancel
// large terms when L is large on the nonzeros).  Terms are summed in fp64.

#include <climits>

#include "tile.h"

namespace nmd {

// Per workgroup: partial[k * gridDim.x + workgroup] = its share of sum k (k = 0 only, or 0..4
// in the metrics variant).
template <int RP, bool METRICS>
__global__ __launch_bounds__(256) void objective_kernel(
    const float* __restrict__ X, int64_t rows, const float* __restrict__ P,
    const int64_t* __restrict__ cbounds, int nsub, const int64_t* __restrict__ rowptr,
    const int32_t* __restrict__ idx, const float* __restrict__ val, int64_t row_tiles,
    double* __restrict__ partial) {
  constexpr int MI = DenseCfg<RP>::MI;
  constexpr int NT = DenseCfg<RP>::NT;
  constexpr int NQ = METRICS ? 5 : 1;
  __shared__ __attribute__((aligned(16))) float tile[NT * (RP + 4)];
  __shared__ double red[256];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int q = lane >> 4, l16 = lane & 15;

  const int64_t logical = xcd_logical(blockIdx.x, (int64_t)gridDim.x);
  const int64_t unit = logical / row_tiles;
  const int64_t rt = logical - unit * row_tiles;
  const int b = (int)(unit / nsub), s = (int)(unit - (int64_t)b * nsub);
  const int64_t lo = cbounds[b], len = cbounds[b + 1] - lo;
  const int64_t jb0 = lo + (int64_t)s * len / nsub;
  const int64_t jb1 = lo + (int64_t)(s + 1) * len / nsub;
  const int64_t row0 = rt * (64 * MI) + (int64_t)wave * (16 * MI);

  float a[MI][RP / 4];
  load_x_frags<RP, MI>(a, X, rows, row0, q, l16);

  // Row walks: first entry of row i in column block b at or after column jb0.
  int64_t ptr[MI], end[MI];
  int nextc[MI];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
    const int64_t row = row0 + 16 * mi + l16;
    ptr[mi] = end[mi] = 0;
    nextc[mi] = INT_MAX;
    if (row < rows) {
      int64_t l = rowptr[(int64_t)b * (rows + 1) + row];
      int64_t h = rowptr[(int64_t)b * (rows + 1) + row + 1];
      end[mi] = h;
      while (l < h) {
        const int64_t mid = (l + h) >> 1;
        if (idx[mid] < jb0) l = mid + 1; else h = mid;
      }
      ptr[mi] = l;
      if (l < end[mi]) nextc[mi] = idx[l];
    }
  }

  double acc = 0.0;                            // q0, or f^2 ||S||^2 when !METRICS
  double qs = 0.0, qr = 0.0, qmin = 0.0, qmax = 0.0;  // q1 .. q4
  PanelTile<RP, NT> pt;
  if (jb0 < jb1) pt.fetch(P, jb0, jb1, tid);
  for (int64_t j0 = jb0; j0 < jb1; j0 += NT) {
    __syncthreads();
    pt.stash(tile, tid);
    __syncthreads();
    if (j0 + NT < jb1) pt.fetch(P, j0 + NT, jb1, tid);
    const int left = (int)((jb1 - j0 + 15) / 16);
    const int njb = left < NT / 16 ? left : NT / 16;
    for (int jb = 0; jb < njb; ++jb) {
      floatx4 lt[MI];
      float4 pre[l_lookahead<RP>()];
      float unused[1][RP / 16];
      l_prefetch<RP>(pre, tile, jb, q, l16);
      l_tile<RP, MI, 0>(lt, a, pre, unused, tile, jb, q, l16);
      const int64_t c0 = j0 + 16 * jb + 4 * q;
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) {
        float sv[4] = {0.f, 0.f, 0.f, 0.f};
        bool hit[4] = {false, false, false, false};
        while (nextc[mi] < c0 + 4 && nextc[mi] < jb1) {
          if (nextc[mi] >= c0) {
            const int v = (int)(nextc[mi] - c0);
            const float sval = val[ptr[mi]];
#pragma unroll
            for (int u = 0; u < 4; ++u)
              if (v == u) {
                sv[u] = sval;
                hit[u] = true;
              }
          }
          ++ptr[mi];
          nextc[mi] = ptr[mi] < end[mi] ? idx[ptr[mi]] : INT_MAX;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float l = lt[mi][u];
          const double p = (double)fmaxf(l, 0.f);
          if (hit[u]) {
            const double sd = (double)sv[u];
            const double d = sd - (double)l;
            if constexpr (METRICS) {
              const double e = sd - p;
              qs += d * d;
              qr += e * e;
              qmin += fmin(sd, p);
              qmax += fmax(sd, p);
            } else {
              acc += d * d;
            }
          } else {
            acc += p * p;
            if constexpr (METRICS) qmax += p;
          }
        }
      }
    }
  }

  const double mine[5] = {acc, qs, qr, qmin, qmax};
#pragma unroll
  for (int k = 0; k < NQ; ++k) {
    red[tid] = mine[k];
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
      if (tid < h) red[tid] += red[tid + h];
      __syncthreads();
    }
    if (tid == 0) partial[(int64_t)k * gridDim.x + logical] = red[0];
    __syncthreads();
  }
}

template <int RP>
static hipError_t launch_objective_t(const float* X, int64_t rows, const float* P,
                                     const int64_t* cbounds, int nblk, int nsub,
                                     const int64_t* rowptr, const int32_t* idx, const float* val,
                                     bool metrics, double* partial, int64_t* npartial,
                                     hipStream_t st) {
  const int64_t row_tiles = (rows + rows_per_wg<RP>() - 1) / rows_per_wg<RP>();
  const int64_t total = row_tiles * nblk * nsub;
  *npartial = total;
  if (total <= 0) return hipSuccess;
  if (total > 0x7fffffffLL) return hipErrorInvalidValue;
  if (metrics)
    hipLaunchKernelGGL((objective_kernel<RP, true>), dim3((unsigned)total), dim3(256), 0, st, X,
                       rows, P, cbounds, nsub, rowptr, idx, val, row_tiles, partial);
  else
    hipLaunchKernelGGL((objective_kernel<RP, false>), dim3((unsigned)total), dim3(256), 0, st, X,
                       rows, P, cbounds, nsub, rowptr, idx, val, row_tiles, partial);
  return hipGetLastError();
}

hipError_t launch_objective(const float* X, int64_t rows, const float* P, const int64_t* cbounds,
                            int nblk, int nsub, const int64_t* rowptr, const int32_t* idx,
                            const float* val, int rp, bool metrics, double* partial,
                            int64_t* npartial, hipStream_t st) {
#define CALL(R)                                                                                \
  launch_objective_t<R>(X, rows, P, cbounds, nblk, nsub, rowptr, idx, val, metrics, partial, \
                        npartial, st)
  NMD_RP_DISPATCH(rp, CALL)
#undef CALL
}

}  // namespace nmd
