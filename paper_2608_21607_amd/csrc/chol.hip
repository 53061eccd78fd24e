// The r x r solve of every update through a Cholesky factorisation, on fp64 MFMA.
//
// The least-squares step needs (P_J^T P_J)^-1 (eqs. lsqA, lsqA_sto).  With G = P_J^T P_J
// symmetric positive definite, G = L L^T (Cholesky), and G^-1 = M^T M with M = L^-1.  The
// apply multiplies by -G^-1 as one matrix product, so that is what is formed here:
//
//   1. L by blocks of NB columns, left-looking: launch k has one workgroup per block row
//      i >= k.  Each computes the updated diagonal block A_kk - sum_{l<k} L_kl L_kl^T, factors
//      it (every workgroup of the launch does so, which removes any dependence between them),
//      forms D_k = L_kk^-1 and, for i > k, L_ik = (A_ik - sum_{l<k} L_il L_kl^T) D_k^T.
//   2. M = L^-1 by block columns (one workgroup each): M_jj = D_j and, for i > j,
//      M_ij = -D_i sum_{l=j}^{i-1} L_il M_lj.
//   3. -G^-1 = -M^T M by 64 x 64 tiles: tile (a, b) = -sum_{l >= max(a, b)} M_la^T M_lb.
//
// The launches take a batch of matrices (blockIdx.y), each with its own work area and step id.
// A second form (chol_fused_kernel) runs all three steps for a matrix in one workgroup, the
// diagonal block factored once per block column: one launch per batch, slower on an idle GPU
// but with far fewer launches to queue behind the contraction's workgroups.  A pivot that is
// not positive (or not finite) flags that step as not positive definite; its apply and the
// later ones then write nothing.  Blocks of NB x NB doubles are staged in LDS with row stride
// NB + 1; fp64 MFMA v_mfma_f64_16x16x4f64: srcA lane l = A[l % 16][l / 16], srcB lane
// l = B[l / 16][l % 16], accumulator register v of lane l = D[4 v + l / 16][l % 16].

#include "nmd_internal.h"

namespace nmd {

typedef double dx4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int kThreads = 1024;

// Work area of matrix b: L, M = L^-1, -G^-1 (rp x rp each) and the diagonal blocks D_k.
struct Work {
  double *L, *M, *Gneg, *D;
  __host__ __device__ Work(double* base, int64_t per, int b, int rp) {
    double* w = base + per * b;
    L = w;
    M = w + (int64_t)rp * rp;
    Gneg = w + 2 * (int64_t)rp * rp;
    D = w + 3 * (int64_t)rp * rp;
  }
};

// Copies the NB x NB block at (bi, bj) of a row-major matrix with leading dimension ld into LDS.
template <int NB>
__device__ __forceinline__ void stage(double* dst, const double* __restrict__ src, int ld, int bi,
                                      int bj) {
  constexpr int LS = NB + 1;
  for (int e = threadIdx.x; e < NB * NB; e += kThreads) {
    const int r = e / NB, c = e - r * NB;
    dst[r * LS + c] = src[(int64_t)(bi * NB + r) * ld + bj * NB + c];
  }
}

// acc += A B^T for two NB x NB blocks in LDS: (A B^T)[r][c] = sum_m A[r][m] B[c][m]; wave w
// owns the 16 x 16 output sub-tile (w / (NB / 16), w % (NB / 16)).
template <int NB>
__device__ __forceinline__ void mma_abt(dx4& acc, const double* A, const double* B, int ri,
                                        int ci, int q, int l16) {
  constexpr int LS = NB + 1;
#pragma unroll 4
  for (int m0 = 0; m0 < NB; m0 += 4) {
    const double a = A[(16 * ri + l16) * LS + m0 + q];
    const double b = B[(16 * ci + l16) * LS + m0 + q];
    acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc, 0, 0, 0);
  }
}

// acc += A^T B: (A^T B)[r][c] = sum_m A[m][r] B[m][c].
template <int NB>
__device__ __forceinline__ void mma_atb(dx4& acc, const double* A, const double* B, int ri,
                                        int ci, int q, int l16) {
  constexpr int LS = NB + 1;
#pragma unroll 4
  for (int m0 = 0; m0 < NB; m0 += 4) {
    const double a = A[(m0 + q) * LS + 16 * ri + l16];
    const double b = B[(m0 + q) * LS + 16 * ci + l16];
    acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc, 0, 0, 0);
  }
}

// acc += A B: (A B)[r][c] = sum_m A[r][m] B[m][c].
template <int NB>
__device__ __forceinline__ void mma_ab(dx4& acc, const double* A, const double* B, int ri, int ci,
                                       int q, int l16) {
  constexpr int LS = NB + 1;
#pragma unroll 4
  for (int m0 = 0; m0 < NB; m0 += 4) {
    const double a = A[(16 * ri + l16) * LS + m0 + q];
    const double b = B[(m0 + q) * LS + 16 * ci + l16];
    acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc, 0, 0, 0);
  }
}

// Writes s * acc (the wave's sub-tile) into an LDS block.
template <int NB>
__device__ __forceinline__ void put_tile(double* dst, const dx4& acc, double s, int ri, int ci,
                                         int q, int l16) {
  constexpr int LS = NB + 1;
#pragma unroll
  for (int v = 0; v < 4; ++v) dst[(16 * ri + 4 * v + q) * LS + 16 * ci + l16] = s * acc[v];
}

// 1 / x to full double precision: the fp32 reciprocal estimate refined by two Newton steps
// (each doubles the correct bits: 2^-23 -> 2^-46 -> beyond 2^-53); a plain division where x is
// outside the range the fp32 estimate covers.
__device__ __forceinline__ double recip(double x) {
  if (!(x > 1e-30 && x < 1e30)) return 1.0 / x;  // outside the fp32 estimate's range
  double y = (double)(1.0f / (float)x);
  y = y * (2.0 - x * y);
  return y * (2.0 - x * y);
}

// In-place Cholesky of the NB x NB block in LDS (lower triangle) and D = L^-1 into `inv`, in one
// elimination: step j removes (a_rj / a_jj) times row j from every row r > j, in the columns
// right of j of A (the trailing update) and in the columns up to j of E (which starts as I).  So
// E A = U with U upper triangular and E unit lower triangular; with p_j = a_jj at step j,
// L[r][c] = a_rc / sqrt(p_c) and L^-1 = diag(1 / sqrt(p)) E.  Thread t owns row t / (NB / 4) and
// columns (t % (NB / 4)) + (NB / 4) u, u = 0..3, of both.  Step j reads column j of A and row j
// of E, which no thread writes in that step, so one barrier per step suffices.  Returns false if
// a pivot was not positive (or not finite).
template <int NB>
__device__ bool factor_block(double* A, double* inv) {
  constexpr int LS = NB + 1;
  constexpr int TPR = NB / 4;
  const int tid = threadIdx.x;
  const bool act = tid < NB * TPR;
  const int r = act ? tid / TPR : 0;
  const int c0 = act ? tid % TPR : 0;
  if (act) {
#pragma unroll
    for (int u = 0; u < 4; ++u) inv[r * LS + c0 + TPR * u] = (r == c0 + TPR * u) ? 1.0 : 0.0;
  }
  bool ok = true;
  __syncthreads();
  for (int j = 0; j < NB; ++j) {
    double piv = A[j * LS + j];
    if (!(piv > 0.0) || !isfinite(piv)) {
      ok = false;
      piv = 1.0;
    }
    if (act && r > j) {
      const double f = A[r * LS + j] * recip(piv);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = c0 + TPR * u;
        if (c > j) {
          if (c <= r) A[r * LS + c] -= f * A[c * LS + j];
        } else {
          inv[r * LS + c] -= f * inv[j * LS + c];
        }
      }
    }
    __syncthreads();
  }
  // L[r][c] = a_rc / sqrt(p_c) (zero above the diagonal), L^-1[r][c] = E[r][c] / sqrt(p_r)
  double lv[4], dv[4];
  if (act) {
    double pr = A[r * LS + r];
    pr = (pr > 0.0 && isfinite(pr)) ? pr : 1.0;
    const double sr = 1.0 / sqrt(pr);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = c0 + TPR * u;
      double pc = A[c * LS + c];
      pc = (pc > 0.0 && isfinite(pc)) ? pc : 1.0;
      lv[u] = c <= r ? A[r * LS + c] / sqrt(pc) : 0.0;
      dv[u] = c <= r ? inv[r * LS + c] * sr : 0.0;
    }
  }
  __syncthreads();
  if (act) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      A[r * LS + c0 + TPR * u] = lv[u];
      inv[r * LS + c0 + TPR * u] = dv[u];
    }
  }
  __syncthreads();
  return ok;
}

}  // namespace

// Launch k of step 1: block row i = k + blockIdx.x of matrix blockIdx.y.
template <int NB>
__global__ __launch_bounds__(kThreads) void chol_col_kernel(const double* __restrict__ Gall,
                                                            double* __restrict__ work,
                                                            int64_t per, int rp, int k,
                                                            int* status, SolveBatch sb) {
  constexpr int LS = NB + 1;
  constexpr int NT = NB / 16;  // sub-tiles per dimension
  __shared__ double sA[NB * LS], sB[NB * LS], s1[NB * LS], s2[NB * LS];
  const Work wk(work, per, blockIdx.y, rp);
  const double* __restrict__ G = Gall + (int64_t)blockIdx.y * rp * rp;
  double* __restrict__ L = wk.L;
  double* __restrict__ D = wk.D;
  const int i = k + blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane >> 4, l16 = lane & 15;
  const bool mw = wave < NT * NT;  // waves with an output sub-tile
  const int ri = wave / NT, ci = wave % NT;
  dx4 akk = {0.0, 0.0, 0.0, 0.0}, aik = {0.0, 0.0, 0.0, 0.0};
  for (int l = 0; l < k; ++l) {
    __syncthreads();
    stage<NB>(s1, L, rp, k, l);
    if (i != k) stage<NB>(s2, L, rp, i, l);
    __syncthreads();
    if (mw) {
      mma_abt<NB>(akk, s1, s1, ri, ci, q, l16);
      if (i != k) mma_abt<NB>(aik, s2, s1, ri, ci, q, l16);
    }
  }
  stage<NB>(sA, G, rp, k, k);
  if (i != k) stage<NB>(sB, G, rp, i, k);
  __syncthreads();
  if (mw) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int o = (16 * ri + 4 * v + q) * LS + 16 * ci + l16;
      sA[o] -= akk[v];
      if (i != k) sB[o] -= aik[v];
    }
  }
  const bool ok = factor_block<NB>(sA, s1);  // s1 = D_k = L_kk^-1
  if (!ok && blockIdx.x == 0 && threadIdx.x == 0)
    flag_status(status, STATUS_NOTPD, sb.step_id[blockIdx.y]);
  if (i == k) {
    for (int e = threadIdx.x; e < NB * NB; e += kThreads) {
      const int r = e / NB, c = e - r * NB;
      L[(int64_t)(k * NB + r) * rp + k * NB + c] = sA[r * LS + c];
      D[(int64_t)k * NB * NB + e] = s1[r * LS + c];
    }
    return;
  }
  // L_ik = A_ik D_k^T
  dx4 o = {0.0, 0.0, 0.0, 0.0};
  if (mw) mma_abt<NB>(o, sB, s1, ri, ci, q, l16);
  if (mw) {
#pragma unroll
    for (int v = 0; v < 4; ++v)
      L[(int64_t)(i * NB + 16 * ri + 4 * v + q) * rp + k * NB + 16 * ci + l16] = o[v];
  }
}

// Step 2 for block column j of M = L^-1 (rows i >= j): M_jj = D_j and, for i > j,
// M_ij = -D_i sum_{l=j}^{i-1} L_il M_lj.  Four NB x NB LDS blocks; ends with the LDS free once
// the caller synchronises.
template <int NB>
__device__ void trinv_column(const double* __restrict__ L, const double* __restrict__ D,
                             double* __restrict__ Mb, int rp, int j, double* sL, double* sM,
                             double* sT, double* sD) {
  constexpr int LS = NB + 1;
  constexpr int NT = NB / 16;
  const int nb = rp / NB;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane >> 4, l16 = lane & 15;
  const bool mw = wave < NT * NT;
  const int ri = wave / NT, ci = wave % NT;
  for (int e = threadIdx.x; e < NB * NB; e += kThreads) {
    const int r = e / NB, c = e - r * NB;
    Mb[(int64_t)(j * NB + r) * rp + j * NB + c] = D[(int64_t)j * NB * NB + e];
  }
  for (int i = j + 1; i < nb; ++i) {
    dx4 t = {0.0, 0.0, 0.0, 0.0};
    for (int l = j; l < i; ++l) {
      __syncthreads();  // Mb writes of the previous block row are visible; LDS is free
      stage<NB>(sL, L, rp, i, l);
      stage<NB>(sM, Mb, rp, l, j);
      __syncthreads();
      if (mw) mma_ab<NB>(t, sL, sM, ri, ci, q, l16);
    }
    __syncthreads();
    if (mw) put_tile<NB>(sT, t, 1.0, ri, ci, q, l16);
    for (int e = threadIdx.x; e < NB * NB; e += kThreads) {
      const int r = e / NB, c = e - r * NB;
      sD[r * LS + c] = D[(int64_t)i * NB * NB + e];
    }
    __syncthreads();
    dx4 o = {0.0, 0.0, 0.0, 0.0};
    if (mw) mma_ab<NB>(o, sD, sT, ri, ci, q, l16);
    if (mw) {
#pragma unroll
      for (int v = 0; v < 4; ++v)
        Mb[(int64_t)(i * NB + 16 * ri + 4 * v + q) * rp + j * NB + 16 * ci + l16] = -o[v];
    }
  }
}

// Step 2: block column j = blockIdx.x of matrix blockIdx.y.
template <int NB>
__global__ __launch_bounds__(kThreads) void chol_trinv_kernel(double* __restrict__ work,
                                                              int64_t per, int rp) {
  constexpr int LS = NB + 1;
  __shared__ double sL[NB * LS], sM[NB * LS], sT[NB * LS], sD[NB * LS];
  const Work wk(work, per, blockIdx.y, rp);
  trinv_column<NB>(wk.L, wk.D, wk.M, rp, blockIdx.x, sL, sM, sT, sD);
}

// Step 3 for tile (a, b), a <= b, of -G^-1 = -M^T M: -sum_{l >= b} M_la^T M_lb, written to
// both (a, b) and (b, a).  Two NB x NB LDS blocks.
template <int NB>
__device__ void gram_tile(const double* __restrict__ Mb, double* __restrict__ Gneg, int rp, int a,
                          int b, double* s1, double* s2) {
  constexpr int NT = NB / 16;
  const int nb = rp / NB;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane >> 4, l16 = lane & 15;
  const bool mw = wave < NT * NT;
  const int ri = wave / NT, ci = wave % NT;
  dx4 acc = {0.0, 0.0, 0.0, 0.0};
  for (int l = b; l < nb; ++l) {
    __syncthreads();
    stage<NB>(s1, Mb, rp, l, a);
    stage<NB>(s2, Mb, rp, l, b);
    __syncthreads();
    if (mw) mma_atb<NB>(acc, s1, s2, ri, ci, q, l16);
  }
  if (mw) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int r = 16 * ri + 4 * v + q, c = 16 * ci + l16;
      Gneg[(int64_t)(a * NB + r) * rp + b * NB + c] = -acc[v];
      if (a != b) Gneg[(int64_t)(b * NB + c) * rp + a * NB + r] = -acc[v];
    }
  }
}

// Pair index p -> tile (a, b) with a <= b, in the order (0,0), (0,1), ..., (1,1), ...
__device__ __forceinline__ void tile_pair(int p, int nb, int& a, int& b) {
  a = 0;
  while (p >= nb - a) {
    p -= nb - a;
    ++a;
  }
  b = a + p;
}

// Step 3: tile pair blockIdx.x of matrix blockIdx.y.
template <int NB>
__global__ __launch_bounds__(kThreads) void chol_gram_kernel(double* __restrict__ work,
                                                             int64_t per, int rp,
                                                             const int* status, SolveBatch sb) {
  constexpr int LS = NB + 1;
  __shared__ double s1[NB * LS], s2[NB * LS];
  const Work wk(work, per, blockIdx.y, rp);
  int a, b;
  tile_pair(blockIdx.x, rp / NB, a, b);
  if (step_blocked(status, sb.step_id[blockIdx.y])) return;  // its apply writes nothing
  gram_tile<NB>(wk.M, wk.Gneg, rp, a, b, s1, s2);
}

// Steps 1-3 for matrix blockIdx.x by a single workgroup: L by block columns (the diagonal
// block factored once per column, then the blocks below it), M = L^-1 by block columns, then
// the tiles of -M^T M.  One launch per batch instead of one per block column and two more; a
// batch's matrices run on separate CUs.
template <int NB>
__global__ __launch_bounds__(kThreads) void chol_fused_kernel(const double* __restrict__ Gall,
                                                              double* __restrict__ work,
                                                              int64_t per, int rp, int* status,
                                                              SolveBatch sb) {
  constexpr int LS = NB + 1;
  constexpr int NT = NB / 16;
  __shared__ double s0[NB * LS], s1[NB * LS], s2[NB * LS], s3[NB * LS];
  const Work wk(work, per, blockIdx.x, rp);
  const double* __restrict__ G = Gall + (int64_t)blockIdx.x * rp * rp;
  double* __restrict__ L = wk.L;
  double* __restrict__ D = wk.D;
  const int nb = rp / NB;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q = lane >> 4, l16 = lane & 15;
  const bool mw = wave < NT * NT;
  const int ri = wave / NT, ci = wave % NT;
  bool all_ok = true;
  for (int k = 0; k < nb; ++k) {
    // L_kk and D_k = L_kk^-1 from A_kk - sum_{l<k} L_kl L_kl^T
    dx4 akk = {0.0, 0.0, 0.0, 0.0};
    for (int l = 0; l < k; ++l) {
      __syncthreads();
      stage<NB>(s1, L, rp, k, l);
      __syncthreads();
      if (mw) mma_abt<NB>(akk, s1, s1, ri, ci, q, l16);
    }
    __syncthreads();
    stage<NB>(s0, G, rp, k, k);
    __syncthreads();
    if (mw) {
#pragma unroll
      for (int v = 0; v < 4; ++v) s0[(16 * ri + 4 * v + q) * LS + 16 * ci + l16] -= akk[v];
    }
    const bool ok = factor_block<NB>(s0, s3);  // s0 = L_kk, s3 = D_k (kept for the column)
    all_ok = all_ok && ok;
    for (int e = threadIdx.x; e < NB * NB; e += kThreads) {
      const int r = e / NB, c = e - r * NB;
      L[(int64_t)(k * NB + r) * rp + k * NB + c] = s0[r * LS + c];
      D[(int64_t)k * NB * NB + e] = s3[r * LS + c];
    }
    // L_ik = (A_ik - sum_{l<k} L_il L_kl^T) D_k^T for the blocks below
    for (int i = k + 1; i < nb; ++i) {
      dx4 aik = {0.0, 0.0, 0.0, 0.0};
      for (int l = 0; l < k; ++l) {
        __syncthreads();
        stage<NB>(s1, L, rp, k, l);
        stage<NB>(s2, L, rp, i, l);
        __syncthreads();
        if (mw) mma_abt<NB>(aik, s2, s1, ri, ci, q, l16);
      }
      __syncthreads();
      stage<NB>(s2, G, rp, i, k);
      __syncthreads();
      if (mw) {
#pragma unroll
        for (int v = 0; v < 4; ++v) s2[(16 * ri + 4 * v + q) * LS + 16 * ci + l16] -= aik[v];
      }
      __syncthreads();
      dx4 o = {0.0, 0.0, 0.0, 0.0};
      if (mw) mma_abt<NB>(o, s2, s3, ri, ci, q, l16);
      if (mw) {
#pragma unroll
        for (int v = 0; v < 4; ++v)
          L[(int64_t)(i * NB + 16 * ri + 4 * v + q) * rp + k * NB + 16 * ci + l16] = o[v];
      }
    }
    __syncthreads();  // L of this block column is visible to every wave
  }
  if (!all_ok) {
    if (threadIdx.x == 0) flag_status(status, STATUS_NOTPD, sb.step_id[blockIdx.x]);
    return;  // uniform: every thread saw the same pivots
  }
  for (int j = 0; j < nb; ++j) {
    trinv_column<NB>(L, D, wk.M, rp, j, s0, s1, s2, s3);
    __syncthreads();
  }
  for (int p = 0; p < nb * (nb + 1) / 2; ++p) {
    int a, b;
    tile_pair(p, nb, a, b);
    gram_tile<NB>(wk.M, wk.Gneg, rp, a, b, s0, s1);
    __syncthreads();
  }
}

int64_t chol_work_doubles(int rp) {
  const int NB = rp < 64 ? rp : 64;
  return 3 * (int64_t)rp * rp + (int64_t)(rp / NB) * NB * NB;
}

hipError_t launch_chol_inverse(const double* G, double* work, int rp, int* status,
                               const SolveBatch& sb, double** result, hipStream_t st) {
  if (sb.n < 1 || sb.n > kSolveBatch) return hipErrorInvalidValue;
  const int NB = rp < 64 ? rp : 64;
  const int nb = rp / NB;
  const int64_t per = chol_work_doubles(rp);
  const unsigned nm = (unsigned)sb.n;
#define CHOL_NB(B)                                                                           \
  case B: {                                                                                  \
    for (int k = 0; k < nb; ++k) {                                                           \
      hipLaunchKernelGGL((chol_col_kernel<B>), dim3(nb - k, nm), dim3(kThreads), 0, st, G, work, \
                         per, rp, k, status, sb);                                            \
      hipError_t e = hipGetLastError();                                                      \
      if (e != hipSuccess) return e;                                                         \
    }                                                                                        \
    hipLaunchKernelGGL((chol_trinv_kernel<B>), dim3(nb, nm), dim3(kThreads), 0, st, work, per, \
                       rp);                                                                  \
    hipError_t e = hipGetLastError();                                                        \
    if (e != hipSuccess) return e;                                                           \
    hipLaunchKernelGGL((chol_gram_kernel<B>), dim3(nb * (nb + 1) / 2, nm), dim3(kThreads), 0, st, \
                       work, per, rp, status, sb);                                           \
    break;                                                                                   \
  }
  switch (NB) {
    CHOL_NB(16)
    CHOL_NB(32)
    CHOL_NB(48)
    CHOL_NB(64)
    default: return hipErrorInvalidValue;
  }
#undef CHOL_NB
  for (int b = 0; b < sb.n; ++b) result[b] = Work(work, per, b, rp).Gneg;
  return hipGetLastError();
}

hipError_t launch_chol_inverse_fused(const double* G, double* work, int rp, int* status,
                                     const SolveBatch& sb, double** result, hipStream_t st) {
  if (sb.n < 1 || sb.n > kSolveBatch) return hipErrorInvalidValue;
  const int NB = rp < 64 ? rp : 64;
  const int64_t per = chol_work_doubles(rp);
  const dim3 grid((unsigned)sb.n);
  switch (NB) {
    case 16: hipLaunchKernelGGL((chol_fused_kernel<16>), grid, dim3(kThreads), 0, st, G, work, per, rp, status, sb); break;
    case 32: hipLaunchKernelGGL((chol_fused_kernel<32>), grid, dim3(kThreads), 0, st, G, work, per, rp, status, sb); break;
    case 48: hipLaunchKernelGGL((chol_fused_kernel<48>), grid, dim3(kThreads), 0, st, G, work, per, rp, status, sb); break;
    case 64: hipLaunchKernelGGL((chol_fused_kernel<64>), grid, dim3(kThreads), 0, st, G, work, per, rp, status, sb); break;
    default: return hipErrorInvalidValue;
  }
  for (int b = 0; b < sb.n; ++b) result[b] = Work(work, per, b, rp).Gneg;
  return hipGetLastError();
}

}  // namespace nmd
