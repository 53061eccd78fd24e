// The r x r least-squares solve of every update (eqs. lsqA, lsqA_sto), on the device, in fp64.
//
//   1. Gram matrix G = P_J^T P_J of the panel rows of the block (fp32 inputs, products exact in
//      fp64, sums in fp64), computed in row chunks by many workgroups and reduced in a fixed
//      order (deterministic).  Padded columns (beyond r) are zero, so their diagonal is set to 1.
//   2. G^-1 by block sweeps (in-place Gauss-Jordan elimination by pivot blocks of 64): sweeping
//      pivot block k maps [[P, Q], [Q^T, T]] to [[-P^-1, P^-1 Q], [Q^T P^-1, T - Q^T P^-1 Q]];
//      after every block has been swept the matrix holds -G^-1.  For a symmetric positive
//      definite G every pivot (a Schur complement) is positive definite, so no pivoting is
//      needed; a non-positive pivot flags the step as not positive definite.
//   3. Apply: X = (sum of the partial Y) G^-1, then V <- gamma V + eta (X - A), A <- A + V
//      (heavy-ball momentum on eq. lsqA_sto; eta = 1, gamma = 0 gives A <- X).

#include "nmd_internal.h"

namespace nmd {

enum { STATUS_NOTPD = 1, STATUS_NONFINITE = 2 };

// status[0]: flag bits; status[1]: first failing step id.
__device__ __forceinline__ void flag(int* status, int bit, int step_id) {
  atomicOr(&status[0], bit);
  atomicMin(&status[1], step_id);
}

// ---------------------------------------------------------------------------------- Gram --
// grid (npairs, nchunks); tile T = min(64, rp); thread (tx, ty) in 16 x 16 owns the entries
// (ty + 16a, tx + 16b) of the T x T tile.
template <int T>
__global__ __launch_bounds__(256) void gram_kernel(const float* __restrict__ P, int64_t blk, int rp,
                                                   double* __restrict__ Gpart, int nchunks) {
  constexpr int NA = T / 16;
  constexpr int KB = 32;
  __shared__ float si[KB][T + 1];
  __shared__ float sj[KB][T + 1];
  const int nt = rp / T;
  // pair index -> (ti <= tj)
  int pidx = blockIdx.x, ti = 0;
  while (pidx >= nt - ti) {
    pidx -= nt - ti;
    ++ti;
  }
  const int tj = ti + pidx;
  const int c = blockIdx.y;
  const int64_t k0 = (int64_t)c * blk / nchunks, k1 = (int64_t)(c + 1) * blk / nchunks;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  double acc[NA][NA];
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int b = 0; b < NA; ++b) acc[a][b] = 0.0;
  for (int64_t kb = k0; kb < k1; kb += KB) {
    __syncthreads();
    for (int e = threadIdx.x; e < KB * T; e += 256) {
      const int kk = e / T, col = e - kk * T;
      const int64_t k = kb + kk;
      float vi = 0.f, vj = 0.f;
      if (k < k1) {
        vi = P[k * rp + ti * T + col];
        vj = P[k * rp + tj * T + col];
      }
      si[kk][col] = vi;
      sj[kk][col] = vj;
    }
    __syncthreads();
#pragma unroll 4
    for (int kk = 0; kk < KB; ++kk) {
      double xi[NA], xj[NA];
#pragma unroll
      for (int a = 0; a < NA; ++a) xi[a] = (double)si[kk][ty + 16 * a];
#pragma unroll
      for (int b = 0; b < NA; ++b) xj[b] = (double)sj[kk][tx + 16 * b];
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int b = 0; b < NA; ++b) acc[a][b] = fma(xi[a], xj[b], acc[a][b]);
    }
  }
  double* out = Gpart + (int64_t)c * rp * rp;
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int b = 0; b < NA; ++b)
      out[(int64_t)(ti * T + ty + 16 * a) * rp + tj * T + tx + 16 * b] = acc[a][b];
}

// G[i][j] = sum over chunks of the upper-tile partial (mirrored), identity on padded diagonal.
__global__ __launch_bounds__(256) void gram_reduce_kernel(const double* __restrict__ Gpart,
                                                          int nchunks, int r, int rp, int T,
                                                          double* __restrict__ G) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)rp * rp) return;
  const int i = (int)(e / rp), j = (int)(e % rp);
  const bool up = (i / T) <= (j / T);
  const int64_t src = up ? (int64_t)i * rp + j : (int64_t)j * rp + i;
  double s = 0.0;
  for (int c = 0; c < nchunks; ++c) s += Gpart[(int64_t)c * rp * rp + src];
  if (i >= r || j >= r) s = (i == j) ? 1.0 : 0.0;
  G[e] = s;
}

hipError_t launch_gram(const float* P, int64_t blk, int r, int rp, double* Gpart, int nchunks,
                       double* G, hipStream_t st) {
  const int T = rp < 64 ? rp : 64;
  const int nt = rp / T;
  const int npairs = nt * (nt + 1) / 2;
  switch (T) {
    case 16: hipLaunchKernelGGL((gram_kernel<16>), dim3(npairs, nchunks), dim3(256), 0, st, P, blk, rp, Gpart, nchunks); break;
    case 32: hipLaunchKernelGGL((gram_kernel<32>), dim3(npairs, nchunks), dim3(256), 0, st, P, blk, rp, Gpart, nchunks); break;
    case 48: hipLaunchKernelGGL((gram_kernel<48>), dim3(npairs, nchunks), dim3(256), 0, st, P, blk, rp, Gpart, nchunks); break;
    case 64: hipLaunchKernelGGL((gram_kernel<64>), dim3(npairs, nchunks), dim3(256), 0, st, P, blk, rp, Gpart, nchunks); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n = (int64_t)rp * rp;
  hipLaunchKernelGGL(gram_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                     Gpart, nchunks, r, rp, T, G);
  return hipGetLastError();
}

// -------------------------------------------------------------------------- block sweeps --
// Inverse of one NB x NB pivot block by Gauss-Jordan elimination without pivoting (1 WG).
template <int NB>
__global__ __launch_bounds__(256) void pivot_inverse_kernel(const double* __restrict__ G, int rp,
                                                            int k, double* __restrict__ D,
                                                            int* status, int step_id) {
  __shared__ double a[NB][NB + 1];
  __shared__ double colp[NB];
  __shared__ int bad;
  const int tid = threadIdx.x;
  if (tid == 0) bad = 0;
  for (int e = tid; e < NB * NB; e += 256) {
    const int i = e / NB, j = e % NB;
    a[i][j] = G[(int64_t)(k * NB + i) * rp + k * NB + j];
  }
  __syncthreads();
  for (int p = 0; p < NB; ++p) {
    double piv = a[p][p];
    const bool ok = piv > 0.0 && isfinite(piv);
    if (!ok) piv = 1.0;
    __syncthreads();
    if (tid == 0 && !ok) bad = 1;
    for (int i = tid; i < NB; i += 256) colp[i] = a[i][p];
    __syncthreads();
    for (int j = tid; j < NB; j += 256) a[p][j] = (j == p ? 1.0 : a[p][j]) / piv;
    __syncthreads();
    for (int e = tid; e < NB * NB; e += 256) {
      const int i = e / NB, j = e % NB;
      if (i != p) a[i][j] = (j == p ? 0.0 : a[i][j]) - colp[i] * a[p][j];
    }
    __syncthreads();
  }
  // only the first failing step is recorded (a failure leaves later steps skipped)
  if (tid == 0 && bad && *(volatile int*)status == 0) flag(status, STATUS_NOTPD, step_id);
  for (int e = tid; e < NB * NB; e += 256) {
    const int i = e / NB, j = e % NB;
    // symmetrise: the exact inverse of a symmetric block is symmetric
    D[(int64_t)i * NB + j] = 0.5 * (a[i][j] + a[j][i]);
  }
}

// One block sweep over pivot block k; grid (nblk, nblk), one NB x NB output tile per WG.
template <int NB>
__global__ __launch_bounds__(256) void sweep_kernel(const double* __restrict__ Gin,
                                                    double* __restrict__ Gout, int rp, int k,
                                                    const double* __restrict__ D) {
  constexpr int NA = NB / 16;
  __shared__ double s1[NB][NB];
  __shared__ double s2[NB][NB];
  const int tj = blockIdx.x, ti = blockIdx.y;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  auto load = [&](double (*dst)[NB], int bi, int bj) {
    for (int e = tid; e < NB * NB; e += 256) {
      const int i = e / NB, j = e % NB;
      dst[i][j] = Gin[(int64_t)(bi * NB + i) * rp + bj * NB + j];
    }
  };
  auto loadD = [&](double (*dst)[NB]) {
    for (int e = tid; e < NB * NB; e += 256) dst[e / NB][e % NB] = D[e];
  };
  double acc[NA][NA];
  auto matmul = [&](double (*L)[NB], double (*R)[NB]) {
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int b = 0; b < NA; ++b) acc[a][b] = 0.0;
    for (int kk = 0; kk < NB; ++kk) {
      double l[NA], r[NA];
#pragma unroll
      for (int a = 0; a < NA; ++a) l[a] = L[ty + 16 * a][kk];
#pragma unroll
      for (int b = 0; b < NA; ++b) r[b] = R[kk][tx + 16 * b];
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int b = 0; b < NA; ++b) acc[a][b] = fma(l[a], r[b], acc[a][b]);
    }
  };
  auto store = [&](double sign, bool sub) {
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int b = 0; b < NA; ++b) {
        const int64_t o = (int64_t)(ti * NB + ty + 16 * a) * rp + tj * NB + tx + 16 * b;
        Gout[o] = sub ? Gin[o] - acc[a][b] : sign * acc[a][b];
      }
  };
  if (ti == k && tj == k) {
    loadD(s1);
    __syncthreads();
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int b = 0; b < NA; ++b) acc[a][b] = s1[ty + 16 * a][tx + 16 * b];
    store(-1.0, false);
  } else if (ti == k) {
    loadD(s1);
    load(s2, k, tj);
    __syncthreads();
    matmul(s1, s2);
    store(1.0, false);
  } else if (tj == k) {
    load(s1, ti, k);
    loadD(s2);
    __syncthreads();
    matmul(s1, s2);
    store(1.0, false);
  } else {
    load(s1, ti, k);
    loadD(s2);
    __syncthreads();
    matmul(s1, s2);  // T1 = G_ik D
    __syncthreads();
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int b = 0; b < NA; ++b) s1[ty + 16 * a][tx + 16 * b] = acc[a][b];
    load(s2, k, tj);
    __syncthreads();
    matmul(s1, s2);  // T1 G_kj
    store(1.0, true);
  }
}

hipError_t launch_inverse(double* G, double* Gtmp, int rp, int* status, int step_id,
                          double** result, hipStream_t st) {
  const int NB = rp < 64 ? rp : 64;
  const int nblk = rp / NB;
  double* D = Gtmp + (int64_t)rp * rp;  // NB x NB scratch after the ping-pong buffer
  double* bufs[2] = {G, Gtmp};
  int cur = 0;
  for (int k = 0; k < nblk; ++k) {
    switch (NB) {
      case 16: hipLaunchKernelGGL((pivot_inverse_kernel<16>), dim3(1), dim3(256), 0, st, bufs[cur], rp, k, D, status, step_id); break;
      case 32: hipLaunchKernelGGL((pivot_inverse_kernel<32>), dim3(1), dim3(256), 0, st, bufs[cur], rp, k, D, status, step_id); break;
      case 48: hipLaunchKernelGGL((pivot_inverse_kernel<48>), dim3(1), dim3(256), 0, st, bufs[cur], rp, k, D, status, step_id); break;
      case 64: hipLaunchKernelGGL((pivot_inverse_kernel<64>), dim3(1), dim3(256), 0, st, bufs[cur], rp, k, D, status, step_id); break;
      default: return hipErrorInvalidValue;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    switch (NB) {
      case 16: hipLaunchKernelGGL((sweep_kernel<16>), dim3(nblk, nblk), dim3(256), 0, st, bufs[cur], bufs[cur ^ 1], rp, k, D); break;
      case 32: hipLaunchKernelGGL((sweep_kernel<32>), dim3(nblk, nblk), dim3(256), 0, st, bufs[cur], bufs[cur ^ 1], rp, k, D); break;
      case 48: hipLaunchKernelGGL((sweep_kernel<48>), dim3(nblk, nblk), dim3(256), 0, st, bufs[cur], bufs[cur ^ 1], rp, k, D); break;
      case 64: hipLaunchKernelGGL((sweep_kernel<64>), dim3(nblk, nblk), dim3(256), 0, st, bufs[cur], bufs[cur ^ 1], rp, k, D); break;
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    cur ^= 1;
  }
  *result = bufs[cur];
  return hipSuccess;
}

// --------------------------------------------------------------------------------- apply --
// One workgroup per RW = 256 / TX rows.  The fp64 row sums of the partial Y go to LDS; thread
// (tx, ty) computes row ty, columns tx + TX b of X = Ysum (-Gneg), then the momentum update.
template <int RP, int TX>
__global__ __launch_bounds__(256) void apply_kernel(const float* __restrict__ Ypart,
                                                    int64_t y_stride, int nsplit,
                                                    const double* __restrict__ Gneg,
                                                    float* __restrict__ X, float* __restrict__ V,
                                                    int64_t rows, float eta, float gamma,
                                                    const int* status_in, int* status,
                                                    int step_id) {
  constexpr int RW = 256 / TX;
  constexpr int NC = RP / TX;
  __shared__ double ys[RW][RP + 1];
  const int tid = threadIdx.x, tx = tid % TX, ty = tid / TX;
  const bool skip = *(volatile const int*)status_in != 0;
  if (skip) return;  // an earlier step failed: leave the factors as they are
  const int64_t r0 = (int64_t)blockIdx.x * RW;
  for (int e = tid; e < RW * RP; e += 256) {
    const int i = e / RP, c = e % RP;
    const int64_t row = r0 + i;
    double s = 0.0;
    if (row < rows)
      for (int sp = 0; sp < nsplit; ++sp) s += (double)Ypart[(int64_t)sp * y_stride + row * RP + c];
    ys[i][c] = s;
  }
  __syncthreads();
  double acc[NC];
#pragma unroll
  for (int b = 0; b < NC; ++b) acc[b] = 0.0;
  for (int k = 0; k < RP; ++k) {
    const double yv = ys[ty][k];
    const double* g = Gneg + (int64_t)k * RP + tx;
#pragma unroll
    for (int b = 0; b < NC; ++b) acc[b] = fma(yv, g[TX * b], acc[b]);
  }
  const int64_t row = r0 + ty;
  if (row >= rows) return;
  bool bad = false;
#pragma unroll
  for (int b = 0; b < NC; ++b) {
    const int64_t o = row * RP + tx + TX * b;
    const double xnew = -acc[b];
    const double xa = (double)X[o];
    const double v = (double)gamma * (double)V[o] + (double)eta * (xnew - xa);
    const float xf = (float)(xa + v);
    const float vf = (float)v;
    bad |= !isfinite(xf) || !isfinite(vf);
    X[o] = xf;
    V[o] = vf;
  }
  if (bad) flag(status, STATUS_NONFINITE, step_id);
}

hipError_t launch_apply(const float* Ypart, int64_t y_stride, int nsplit, const double* Gneg,
                        float* X, float* V, int64_t rows, int rp, float eta, float gamma,
                        int* status, int step_id, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
#define CASE(R, TXV)                                                                         \
  case R: {                                                                                  \
    const dim3 grid((unsigned)((rows + (256 / TXV) - 1) / (256 / TXV)));                     \
    hipLaunchKernelGGL((apply_kernel<R, TXV>), grid, dim3(256), 0, st, Ypart, y_stride, nsplit, \
                       Gneg, X, V, rows, eta, gamma, status, status, step_id);              \
    break;                                                                                   \
  }
  switch (rp) {
    CASE(16, 16) CASE(32, 16) CASE(48, 16) CASE(64, 16) CASE(128, 16) CASE(192, 16)
    CASE(256, 16) CASE(320, 32) CASE(384, 32) CASE(448, 32) CASE(512, 32)
    default: return hipErrorInvalidValue;
  }
#undef CASE
  return hipGetLastError();
}

}  // namespace nmd
