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
// same transposed layout), a tile's 16-row j-blocks as interleaved accumulator chains.  Each
// lane owns one row i and four columns 4q..4q+3 of every 16-column block, and walks row i's
// nonzeros of the current column block (sorted by column) in step with the tile loop; an entry
// that falls on one of its four columns switches that term from max(0, L)^2 to (S - L)^2.  So
// each term of eq. SLloss is taken once from the same L: nothing is added over all entries and
// subtracted again at the nonzeros (which would cancel large terms when L is large on the
// nonzeros).  Terms are summed in fp64.

#include <climits>

#include "dense_kernel.h"

namespace nmd {

// J-blocks (16 panel rows each) whose L tiles one group computes as interleaved MFMA chains,
// and accumulators per tile, so that every wave keeps about four independent chains: the
// largest divisor of the tile's block count not above max(1, 4 / MI).
template <int RP>
constexpr int obj_jg() {
  constexpr int MI = DenseLaunch<RP>::MI, NJ = DenseLaunch<RP>::NT / 16;
  int g = 4 / MI < 1 ? 1 : 4 / MI;
  if (g > NJ) g = NJ;
  while (NJ % g) --g;
  return g;
}
template <int RP>
constexpr int obj_na() {
  constexpr int c = DenseLaunch<RP>::MI * obj_jg<RP>();
  return c >= 4 ? 1 : 4 / c;
}
template <int RP>
constexpr int obj_la() { return RP / 16 < 2 ? RP / 16 : 2; }

// Running sums and the per-row CSR walks of one lane (rows row0 + 16 mi + l16): acc is q0 (or,
// in the objective-only variant, q0 + q1) and qs, qr, qmin, qmax are q1 .. q4.
template <int MI>
struct ObjState {
  int64_t ptr[MI], end[MI];
  int nextc[MI];
  double acc, qs, qr, qmin, qmax;
};

// First LA k-groups of the panel fragments of the group's j-blocks jbase .. jbase + JG - 1.
template <int RP>
__device__ __forceinline__ void obj_prefetch(float4 (&pre)[obj_la<RP>()][obj_jg<RP>()],
                                             const float* tile, int jbase, int q, int l16) {
#pragma unroll
  for (int jg = 0; jg < obj_jg<RP>(); ++jg) {
    const float* brow = &tile[((jbase + jg) * 16 + l16) * (RP + 4) + 4 * q];
#pragma unroll
    for (int t = 0; t < obj_la<RP>(); ++t) pre[t][jg] = *reinterpret_cast<const float4*>(brow + 16 * t);
  }
}

// Transposed L tiles of the group (layout as in the dense contraction: lt[jg][mi] lane l,
// register v holds L[row0 + 16 mi + l16][(jbase + jg) * 16 + 4q + v]).  The JG * MI * NA
// accumulator chains take the MFMAs round-robin; each k-group first issues the LDS reads of
// the group LA ahead.
template <int RP>
__device__ __forceinline__ void obj_lgroup(
    floatx4 (&lt)[obj_jg<RP>()][DenseLaunch<RP>::MI],
    const float (&a)[DenseLaunch<RP>::MI][RP / 4],
    const float4 (&pre)[obj_la<RP>()][obj_jg<RP>()], const float* tile, int jbase, int q,
    int l16) {
  constexpr int MI = DenseLaunch<RP>::MI, JG = obj_jg<RP>(), NA = obj_na<RP>();
  constexpr int KG = RP / 16, LA = obj_la<RP>(), LS = RP + 4;
  floatx4 acc[NA][JG][MI];
#pragma unroll
  for (int h = 0; h < NA; ++h)
#pragma unroll
    for (int jg = 0; jg < JG; ++jg)
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) acc[h][jg][mi] = floatx4{0.f, 0.f, 0.f, 0.f};
  float4 bf[KG][JG];
#pragma unroll
  for (int t = 0; t < LA; ++t)
#pragma unroll
    for (int jg = 0; jg < JG; ++jg) bf[t][jg] = pre[t][jg];
#pragma unroll
  for (int t = 0; t < KG; ++t) {
    if (t + LA < KG) {
#pragma unroll
      for (int jg = 0; jg < JG; ++jg)
        bf[t + LA][jg] = *reinterpret_cast<const float4*>(
            &tile[((jbase + jg) * 16 + l16) * LS + 4 * q + 16 * (t + LA)]);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int h = (4 * t + c) % NA;
#pragma unroll
      for (int jg = 0; jg < JG; ++jg) {
        const float4 f = bf[t][jg];
        const float bk = c == 0 ? f.x : c == 1 ? f.y : c == 2 ? f.z : f.w;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
          acc[h][jg][mi] =
              __builtin_amdgcn_mfma_f32_16x16x4f32(bk, a[mi][4 * t + c], acc[h][jg][mi], 0, 0, 0);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int jg = 0; jg < JG; ++jg)
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
      lt[jg][mi] = acc[0][jg][mi];
#pragma unroll
      for (int h = 1; h < NA; ++h) lt[jg][mi] += acc[h][jg][mi];
    }
}

// The eq. SLloss terms of the group.  First the lane's nonzeros among its columns (rare): each
// takes its own terms from its L entry and then zeroes that entry, so that the branch-free pass
// over the tile that follows adds max(0, L)^2 (and, for the metrics, max(0, L)) for exactly
// the other entries.  cbase is the lane's first column of the group (4 columns per j-block
// from there, 16 apart); columns at or past jb1 are zero rows of the tile and carry no entry.
template <int RP, bool METRICS>
__device__ __forceinline__ void obj_terms(ObjState<DenseLaunch<RP>::MI>& st,
                                          floatx4 (&lt)[obj_jg<RP>()][DenseLaunch<RP>::MI],
                                          int cbase, int jb1, const int32_t* __restrict__ idx,
                                          const float* __restrict__ val) {
  constexpr int MI = DenseLaunch<RP>::MI, JG = obj_jg<RP>();
  const int cend = cbase + 16 * (JG - 1) + 4;  // past the lane's last column of the group
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
    while (st.nextc[mi] < cend && st.nextc[mi] < jb1) {
      const int off = st.nextc[mi] - cbase;
      if (off >= 0 && (off & 15) < 4) {
        float lf = 0.f;
#pragma unroll
        for (int jg = 0; jg < JG; ++jg)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (off == 16 * jg + v) {
              lf = lt[jg][mi][v];
              lt[jg][mi][v] = 0.f;
            }
        const double sd = (double)val[st.ptr[mi]];
        const double d = sd - (double)lf;
        if constexpr (METRICS) {
          const double p = (double)fmaxf(lf, 0.f);
          const double e = sd - p;
          st.qs += d * d;
          st.qr += e * e;
          st.qmin += fmin(sd, p);
          st.qmax += fmax(sd, p);
        } else {
          st.acc += d * d;
        }
      }
      ++st.ptr[mi];
      st.nextc[mi] = st.ptr[mi] < st.end[mi] ? idx[st.ptr[mi]] : INT_MAX;
    }
  }
#pragma unroll
  for (int jg = 0; jg < JG; ++jg)
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const double p = (double)fmaxf(lt[jg][mi][v], 0.f);
        st.acc = fma(p, p, st.acc);
        if constexpr (METRICS) st.qmax += p;
      }
}

// All groups of one panel tile (first row j0).
template <int RP, bool METRICS>
__device__ __forceinline__ void objective_tile(ObjState<DenseLaunch<RP>::MI>& st,
                                               const float* tile, int j0, int jb1,
                                               const float (&a)[DenseLaunch<RP>::MI][RP / 4],
                                               const int32_t* __restrict__ idx,
                                               const float* __restrict__ val, int q, int l16) {
  constexpr int MI = DenseLaunch<RP>::MI, JG = obj_jg<RP>();
  constexpr int NG = DenseLaunch<RP>::NT / 16 / JG;
  const int left = (jb1 - j0 + 16 * JG - 1) / (16 * JG);
  const int ng = left < NG ? left : NG;
  float4 pre[obj_la<RP>()][JG];
  obj_prefetch<RP>(pre, tile, 0, q, l16);
  for (int g = 0; g < ng; ++g) {
    floatx4 lt[JG][MI];
    obj_lgroup<RP>(lt, a, pre, tile, g * JG, q, l16);
    if (g + 1 < ng) obj_prefetch<RP>(pre, tile, (g + 1) * JG, q, l16);
    obj_terms<RP, METRICS>(st, lt, j0 + 16 * g * JG + 4 * q, jb1, idx, val);
  }
}

// One step of the double-buffered direct pipeline (as in the dense contraction): the restrict
// qualifiers let the compiler read `cur` while the direct loads into `nxt` are in flight.
template <int RP, bool METRICS>
__device__ __forceinline__ void objective_step(
    ObjState<DenseLaunch<RP>::MI>& st, const float* __restrict__ cur, float* __restrict__ nxt,
    const float* __restrict__ P, int j0, int jb1, const float (&a)[DenseLaunch<RP>::MI][RP / 4],
    const int32_t* __restrict__ idx, const float* __restrict__ val, int wave, int lane, int q,
    int l16) {
  if (nxt) issue_tile<RP>(nxt, P, j0 + DenseLaunch<RP>::NT, jb1, wave, lane);
  objective_tile<RP, METRICS>(st, cur, j0, jb1, a, idx, val, q, l16);
}

// Per workgroup: partial[k * gridDim.x + workgroup] = its share of sum k (k = 0 only, or 0..4
// in the metrics variant).  Same launch shapes and panel pipeline as the dense contraction.
template <int RP, bool METRICS>
__global__ __launch_bounds__(64 * DenseLaunch<RP>::WAVES) void objective_kernel(
    const float* __restrict__ X, int64_t rows, const float* __restrict__ P,
    const int64_t* __restrict__ cbounds, int nsub, const int64_t* __restrict__ rowptr,
    const int32_t* __restrict__ idx, const float* __restrict__ val, int64_t row_tiles,
    double* __restrict__ partial) {
  constexpr int MI = DenseLaunch<RP>::MI;
  constexpr int WAVES = DenseLaunch<RP>::WAVES;
  constexpr int NT = DenseLaunch<RP>::NT;
  constexpr bool DIRECT = DenseLaunch<RP>::DIRECT;
  constexpr int LS = RP + 4;
  constexpr int NQ = METRICS ? 5 : 1;
  constexpr int THREADS = 64 * WAVES;
  __shared__ __attribute__((aligned(16))) float smem[(DIRECT ? 2 : 1) * NT * LS];
  __shared__ double red[THREADS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q = lane >> 4, l16 = lane & 15;

  const int64_t logical = xcd_logical(blockIdx.x, (int64_t)gridDim.x);
  const int64_t unit = logical / row_tiles;
  const int64_t rt = logical - unit * row_tiles;
  const int b = (int)(unit / nsub), s = (int)(unit - (int64_t)b * nsub);
  const int64_t lo = cbounds[b], len = cbounds[b + 1] - lo;
  const int jb0 = (int)(lo + (int64_t)s * len / nsub);      // columns < 2^31
  const int jb1 = (int)(lo + (int64_t)(s + 1) * len / nsub);
  const int64_t row0 = rt * dense_rows<RP>() + (int64_t)wave * (16 * MI);

  float a[MI][RP / 4];
  load_x_frags<RP, MI>(a, X, rows, row0, q, l16);

  // Row walks: first entry of row i in column block b at or after column jb0.
  ObjState<MI> st;
  st.acc = st.qs = st.qr = st.qmin = st.qmax = 0.0;
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
    const int64_t row = row0 + 16 * mi + l16;
    st.ptr[mi] = st.end[mi] = 0;
    st.nextc[mi] = INT_MAX;
    if (row < rows) {
      int64_t l = rowptr[(int64_t)b * (rows + 1) + row];
      int64_t h = rowptr[(int64_t)b * (rows + 1) + row + 1];
      st.end[mi] = h;
      while (l < h) {
        const int64_t mid = (l + h) >> 1;
        if (idx[mid] < jb0) l = mid + 1; else h = mid;
      }
      st.ptr[mi] = l;
      if (l < st.end[mi]) st.nextc[mi] = idx[l];
    }
  }

  if constexpr (DIRECT) {
    if (jb0 < jb1) issue_tile<RP>(smem, P, jb0, jb1, wave, lane);
    int cur = 0;
    for (int j0 = jb0; j0 < jb1; j0 += NT, cur ^= 1) {
      __builtin_amdgcn_s_waitcnt(0);  // this wave's loads of the tile have landed
      __syncthreads();                // every wave's have; the other buffer is free again
      float* nxt = j0 + NT < jb1 ? smem + (cur ^ 1) * (NT * LS) : nullptr;
      objective_step<RP, METRICS>(st, smem + cur * (NT * LS), nxt, P, j0, jb1, a, idx, val, wave,
                                  lane, q, l16);
    }
  } else {
    PanelTile<RP, NT, THREADS> pt;
    if (jb0 < jb1) pt.fetch(P, jb0, jb1, tid);
    for (int j0 = jb0; j0 < jb1; j0 += NT) {
      __syncthreads();
      pt.stash(smem, tid);
      __syncthreads();
      if (j0 + NT < jb1) pt.fetch(P, j0 + NT, jb1, tid);
      objective_tile<RP, METRICS>(st, smem, j0, jb1, a, idx, val, q, l16);
    }
  }

  const double mine[5] = {st.acc, st.qs, st.qr, st.qmin, st.qmax};
#pragma unroll
  for (int k = 0; k < NQ; ++k) {
    red[tid] = mine[k];
    __syncthreads();
    for (int h = THREADS / 2; h > 0; h >>= 1) {
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
  const int64_t row_tiles = (rows + dense_rows<RP>() - 1) / dense_rows<RP>();
  const int64_t total = row_tiles * nblk * nsub;
  *npartial = total;
  if (total <= 0) return hipSuccess;
  if (total > 0x7fffffffLL) return hipErrorInvalidValue;
  const dim3 block(64 * DenseLaunch<RP>::WAVES);
  if (metrics)
    hipLaunchKernelGGL((objective_kernel<RP, true>), dim3((unsigned)total), block, 0, st, X,
                       rows, P, cbounds, nsub, rowptr, idx, val, row_tiles, partial);
  else
    hipLaunchKernelGGL((objective_kernel<RP, false>), dim3((unsigned)total), block, 0, st, X,
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
