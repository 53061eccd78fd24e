// The r x r least-squares solve of every update (eqs. lsqA, lsqA_sto), on the device, in fp64.
//
//   1. Gram matrix G = P_J^T P_J of the panel rows of the block (fp32 inputs, products exact in
//      fp64, sums in fp64), computed in row chunks by many workgroups and reduced in a fixed
//      order (deterministic).  Padded columns (beyond r) are zero, so their diagonal is set to 1.
//   2. -G^-1 through the Cholesky factorisation G = L L^T (chol.hip).
//   3. Apply: with U = Delta_{:J} P_J (the sum of the partial outputs), the step is U G^-1
//      (eqs. spLsqA, lsqA_sto), then V <- gamma V + eta U G^-1, A <- A + V (heavy-ball
//      momentum; eta = 1, gamma = 0 gives the exact least-squares update).

#include "nmd_internal.h"

namespace nmd {


typedef double doublex4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------------- Gram --
// grid (npairs, nchunks); tile T = min(64, rp).  A workgroup accumulates the T x T tile
// (ti, tj), ti <= tj, of P^T P over one chunk of panel rows on fp64 MFMA: wave w owns the
// 16-row block w of the tile; srcA lane l = P[k + l/16][ti T + 16 w + l%16], srcB lane l =
// P[k + l/16][tj T + 16 cb + l%16] (fp32 inputs widened exactly to fp64).
template <int T>
__global__ __launch_bounds__(256) void gram_kernel(const float* __restrict__ Pbase, SolveBatch sb,
                                                   int rp, double* __restrict__ Gpart_all,
                                                   int nchunks) {
  // matrix blockIdx.z of the batch: panel rows j0 .. j0 + blk of Pbase, partials at its slot
  const float* __restrict__ P = Pbase + sb.j0[blockIdx.z] * rp;
  const int64_t blk = sb.blk[blockIdx.z];
  double* __restrict__ Gpart = Gpart_all + (int64_t)blockIdx.z * nchunks * rp * rp;
  constexpr int NCB = T / 16;
  constexpr int KB = 64;
  __shared__ float si[KB][T + 1];
  __shared__ float sj[KB][T + 1];
  const int nt = rp / T;
  int pidx = blockIdx.x, ti = 0;  // pair index -> (ti <= tj)
  while (pidx >= nt - ti) {
    pidx -= nt - ti;
    ++ti;
  }
  const int tj = ti + pidx;
  const int c = blockIdx.y;
  const int64_t k0 = (int64_t)c * blk / nchunks, k1 = (int64_t)(c + 1) * blk / nchunks;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q = lane >> 4, l16 = lane & 15;
  const bool active = wave < NCB;
  doublex4 acc[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) acc[cb] = doublex4{0.0, 0.0, 0.0, 0.0};
  for (int64_t kb = k0; kb < k1; kb += KB) {
    __syncthreads();
    for (int e = tid; e < KB * T; e += 256) {
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
    if (active) {
      for (int kk = 0; kk < KB; kk += 4) {
        const double av = (double)si[kk + q][16 * wave + l16];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
          const double bv = (double)sj[kk + q][16 * cb + l16];
          acc[cb] = __builtin_amdgcn_mfma_f64_16x16x4f64(av, bv, acc[cb], 0, 0, 0);
        }
      }
    }
  }
  if (!active) return;
  double* out = Gpart + (int64_t)c * rp * rp;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int v = 0; v < 4; ++v)
      out[(int64_t)(ti * T + 16 * wave + 4 * v + q) * rp + tj * T + 16 * cb + l16] = acc[cb][v];
}

// G[i][j] = sum over chunks of the upper-tile partial (mirrored), identity on padded diagonal.
__global__ __launch_bounds__(256) void gram_reduce_kernel(const double* __restrict__ Gpart_all,
                                                          int nchunks, int r, int rp, int T,
                                                          double* __restrict__ G_all) {
  const double* __restrict__ Gpart = Gpart_all + (int64_t)blockIdx.y * nchunks * rp * rp;
  double* __restrict__ G = G_all + (int64_t)blockIdx.y * rp * rp;
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

hipError_t launch_gram(const float* P, const SolveBatch& sb, int r, int rp, double* Gpart,
                       int nchunks, double* G, hipStream_t st) {
  if (sb.n < 1 || sb.n > kSolveBatch) return hipErrorInvalidValue;
  const int T = rp < 64 ? rp : 64;
  const int nt = rp / T;
  const int npairs = nt * (nt + 1) / 2;
  const dim3 grid(npairs, nchunks, sb.n);
  switch (T) {
    case 16: hipLaunchKernelGGL((gram_kernel<16>), grid, dim3(256), 0, st, P, sb, rp, Gpart, nchunks); break;
    case 32: hipLaunchKernelGGL((gram_kernel<32>), grid, dim3(256), 0, st, P, sb, rp, Gpart, nchunks); break;
    case 48: hipLaunchKernelGGL((gram_kernel<48>), grid, dim3(256), 0, st, P, sb, rp, Gpart, nchunks); break;
    case 64: hipLaunchKernelGGL((gram_kernel<64>), grid, dim3(256), 0, st, P, sb, rp, Gpart, nchunks); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t n = (int64_t)rp * rp;
  hipLaunchKernelGGL(gram_reduce_kernel, dim3((unsigned)((n + 255) / 256), sb.n), dim3(256), 0, st,
                     Gpart, nchunks, r, rp, T, G);
  return hipGetLastError();
}

// --------------------------------------------------------------------------------- apply --
// U for rows r0 .. r0 + RW - 1: the fp64 sums of the nsplit partial outputs (and of Ysp when not
// NULL), stored into the LDS tile ys (row stride LS) as T.  Each thread owns NE float4 groups,
// taken EC (at most 8) at a time; the EC loads of one partial are issued before any is used, so
// a thread waits for one round trip per partial and chunk rather than one per group.
template <int RP, int RW, int LS, typename T>
__device__ __forceinline__ void stage_u(T* ys, const float* __restrict__ Ypart, int64_t y_stride,
                                        int nsplit, const float* __restrict__ Ysp, int64_t r0,
                                        int64_t rows, int tid) {
  constexpr int NE = RW * RP / 4 / 256;
  constexpr int EC = NE <= 8 ? NE : (NE % 8 == 0 ? 8 : (NE % 7 == 0 ? 7 : (NE % 6 == 0 ? 6 : 5)));
  static_assert(NE >= 1 && NE * 256 == RW * RP / 4 && NE % EC == 0, "staging shape");
#pragma unroll
  for (int e0 = 0; e0 < NE; e0 += EC) {
    double s[EC][4];
#pragma unroll
    for (int e = 0; e < EC; ++e) s[e][0] = s[e][1] = s[e][2] = s[e][3] = 0.0;
    // rows past the end read the last row (no branch around the load) and count zero
    auto add = [&](const float* __restrict__ base) {
      float4 v[EC];
#pragma unroll
      for (int e = 0; e < EC; ++e) {
        const int f = tid + 256 * (e0 + e);
        const int i = f / (RP / 4), c4 = f - i * (RP / 4);
        const int64_t row = r0 + i;
        const float4 t =
            *reinterpret_cast<const float4*>(base + (row < rows ? row : rows - 1) * RP + 4 * c4);
        const bool in = row < rows;
        v[e] = make_float4(in ? t.x : 0.f, in ? t.y : 0.f, in ? t.z : 0.f, in ? t.w : 0.f);
      }
#pragma unroll
      for (int e = 0; e < EC; ++e) {
        s[e][0] += (double)v[e].x;
        s[e][1] += (double)v[e].y;
        s[e][2] += (double)v[e].z;
        s[e][3] += (double)v[e].w;
      }
    };
    for (int sp = 0; sp < nsplit; ++sp) add(Ypart + (int64_t)sp * y_stride);
    if (Ysp) add(Ysp);
#pragma unroll
    for (int e = 0; e < EC; ++e) {
      const int f = tid + 256 * (e0 + e);
      const int i = f / (RP / 4), c4 = f - i * (RP / 4);
      T* d = &ys[i * LS + 4 * c4];
      d[0] = (T)s[e][0];
      d[1] = (T)s[e][1];
      d[2] = (T)s[e][2];
      d[3] = (T)s[e][3];
    }
  }
}

// The momentum update of a wave's output elements: element (a, b, v) of lane (q, l16) is row
// r0 + rowof(a) + 4 v + q, column colof(b) + l16, with step = -acc[a][b][v].  X and V are read
// in groups of GU = 2 (a, b) blocks (8 elements per lane), rows past the end clamped to the last
// one, each group's loads issued before the previous group is updated.
template <int RP, int NRB, int NCB, typename RowOf, typename ColOf>
struct MomentumUpdate {
  static constexpr int NU = NRB * NCB;  // (a, b) blocks, u = b * NRB + a
  static constexpr int GU = NU < 2 ? NU : 2;
  static constexpr int NG = (NU + GU - 1) / GU;
  const float* __restrict__ Xin;
  const float* __restrict__ Vin;
  int64_t r0, rows;
  int q, l16;
  RowOf rowof;
  ColOf colof;
  float xv[2][GU][4], vv[2][GU][4];

  __device__ __forceinline__ void load(int grp, int buf) {
#pragma unroll
    for (int g = 0; g < GU; ++g) {
      const int u0 = grp * GU + g;
      const int u = u0 < NU ? u0 : NU - 1;  // a last group may be short
      const int a = u % NRB, b = u / NRB;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        int64_t row = r0 + rowof(a) + 4 * v + q;
        row = row < rows ? row : rows - 1;
        const int64_t o = row * RP + colof(b) + l16;
        xv[buf][g][v] = u0 < NU ? Xin[o] : 0.f;
        vv[buf][g][v] = u0 < NU ? Vin[o] : 0.f;
      }
    }
  }
  // Writes Xout and Vout; returns true if a result was not finite.
  __device__ __forceinline__ bool finish(const doublex4 (&acc)[NRB][NCB], float* __restrict__ Xout,
                                         float* __restrict__ Vout, float eta, float gamma) {
    bool bad = false;
    load(0, 0);
#pragma unroll
    for (int grp = 0; grp < NG; ++grp) {
      if (grp + 1 < NG) load(grp + 1, (grp + 1) & 1);
      const int buf = grp & 1;
#pragma unroll
      for (int g = 0; g < GU; ++g) {
        const int u0 = grp * GU + g;
        if (u0 >= NU) continue;
        const int u = u0 < NU ? u0 : NU - 1;
        const int a = u % NRB, b = u / NRB;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int64_t row = r0 + rowof(a) + 4 * v + q;
          if (row < rows) {
            const int64_t o = row * RP + colof(b) + l16;
            const double stepv = -acc[a][b][v];
            const double vn = (double)gamma * (double)vv[buf][g][v] + (double)eta * stepv;
            const float xf = (float)((double)xv[buf][g][v] + vn);
            const float vf = (float)vn;
            bad |= !isfinite(xf) || !isfinite(vf);
            Xout[o] = xf;
            Vout[o] = vf;
          }
        }
      }
    }
    return bad;
  }
};

template <int RP, int NRB, int NCB, typename RowOf, typename ColOf>
__device__ __forceinline__ MomentumUpdate<RP, NRB, NCB, RowOf, ColOf> momentum_io(
    const float* __restrict__ Xin, const float* __restrict__ Vin, int64_t r0, int64_t rows, int q,
    int l16, RowOf rowof, ColOf colof) {
  MomentumUpdate<RP, NRB, NCB, RowOf, ColOf> m{Xin, Vin, r0, rows, q, l16, rowof, colof, {}, {}};
  return m;
}

template <int RP>
struct ApplyCfg {
  static constexpr int RW = RP <= 64 ? 64 : (RP <= 128 ? 32 : 16);
  static constexpr bool COLS = RP >= 64;                 // waves split columns
  static constexpr int NRB = COLS ? RW / 16 : 1;         // row blocks per wave
  static constexpr int NCB = COLS ? RP / 64 : RP / 16;   // column blocks per wave
};

template <int RP>
__global__ __launch_bounds__(256) void apply_kernel(const float* __restrict__ Ypart,
                                                    int64_t y_stride, int nsplit,
                                                    const float* __restrict__ Ysp,
                                                    const double* __restrict__ Gneg,
                                                    const float* __restrict__ Xin,
                                                    const float* __restrict__ Vin,
                                                    float* __restrict__ Xout,
                                                    float* __restrict__ Vout, int64_t rows,
                                                    float eta, float gamma, int* status,
                                                    int step_id) {
  using C = ApplyCfg<RP>;
  constexpr int RW = C::RW, NRB = C::NRB, NCB = C::NCB;
  constexpr int LS = RP + 1;
  constexpr int PD = 2;  // prefetch distance in k-steps
  __shared__ double ys[RW * LS];
  if (step_blocked(status, step_id)) return;  // this or an earlier step failed: factors stay
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int q = lane >> 4, l16 = lane & 15;
  const int64_t r0 = (int64_t)blockIdx.x * RW;
  stage_u<RP, RW, LS, double>(ys, Ypart, y_stride, nsplit, Ysp, r0, rows, tid);
  __syncthreads();
  auto rblock = [&](int a) { return C::COLS ? a : wave; };
  auto cblock = [&](int b) { return C::COLS ? wave + 4 * b : b; };
  auto io = momentum_io<RP, NRB, NCB>(Xin, Vin, r0, rows, q, l16,
                                      [=](int a) { return 16 * rblock(a); },
                                      [=](int b) { return 16 * cblock(b); });
  doublex4 acc[NRB][NCB];
#pragma unroll
  for (int a = 0; a < NRB; ++a)
#pragma unroll
    for (int b = 0; b < NCB; ++b) acc[a][b] = doublex4{0.0, 0.0, 0.0, 0.0};
  double pre[PD][NCB];
#pragma unroll
  for (int d = 0; d < PD; ++d)
#pragma unroll
    for (int b = 0; b < NCB; ++b)
      pre[d][b] = Gneg[(int64_t)(4 * d + q) * RP + 16 * cblock(b) + l16];
  for (int k0 = 0; k0 < RP; k0 += 4 * PD) {
#pragma unroll
    for (int d = 0; d < PD; ++d) {
      const int k = k0 + 4 * d;
      double bv[NCB];
#pragma unroll
      for (int b = 0; b < NCB; ++b) bv[b] = pre[d][b];
      const int kn = k + 4 * PD;
      if (kn < RP) {
#pragma unroll
        for (int b = 0; b < NCB; ++b) pre[d][b] = Gneg[(int64_t)(kn + q) * RP + 16 * cblock(b) + l16];
      }
#pragma unroll
      for (int a = 0; a < NRB; ++a) {
        const double av = ys[(16 * rblock(a) + l16) * LS + k + q];
#pragma unroll
        for (int b = 0; b < NCB; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f64_16x16x4f64(av, bv[b], acc[a][b], 0, 0, 0);
      }
    }
  }
  const bool bad = io.finish(acc, Xout, Vout, eta, gamma);
  if (bad) flag_status(status, STATUS_NONFINITE, step_id);
}

// Apply for r_p >= 64: a workgroup takes RW rows; each of its 4 waves computes all RW rows for
// a quarter of the columns (column blocks w, w + 4, ...), so G^-1 is read from L2 once per RW
// rows and quarter instead of once per 16 rows.  U (the sum of the partial outputs, formed in
// fp64) is staged in LDS as fp32: it carries fp32 accuracy anyway, and the small tile lets two
// workgroups share a CU, so one's loads overlap the other's MFMAs.  RW is chosen per launch
// (taller tiles need fewer G^-1 reads, but must leave enough workgroups to fill the CUs).
template <int RP, int RW>
struct WideCfg {
  static constexpr int NRB = RW / 16;   // row blocks per wave
  static constexpr int NCB = RP / 64;   // column blocks per wave
};

// Tallest row tile whose accumulators (RW x r_p / 4 doubles per wave) stay within 64 doubles.
template <int RP>
constexpr int wide_max_rw() { return (16384 / RP) >= 64 ? 64 : ((16384 / RP) >= 32 ? 32 : 16); }

template <int RP, int RW>
__global__ __launch_bounds__(256, 2) void apply_wide_kernel(const float* __restrict__ Ypart,
                                                         int64_t y_stride, int nsplit,
                                                         const float* __restrict__ Ysp,
                                                         const double* __restrict__ Gneg,
                                                         const float* __restrict__ Xin,
                                                         const float* __restrict__ Vin,
                                                         float* __restrict__ Xout,
                                                         float* __restrict__ Vout, int64_t rows,
                                                         float eta, float gamma, int* status,
                                                         int step_id) {
  using C = WideCfg<RP, RW>;
  constexpr int NRB = C::NRB, NCB = C::NCB;
  constexpr int LS = RP + 1;
  constexpr int PD = 2;  // prefetch distance in k-steps
  __shared__ float ys[RW * LS];
  if (step_blocked(status, step_id)) return;  // this or an earlier step failed: factors stay
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int q = lane >> 4, l16 = lane & 15;
  const int64_t r0 = (int64_t)blockIdx.x * RW;
  stage_u<RP, RW, LS, float>(ys, Ypart, y_stride, nsplit, Ysp, r0, rows, tid);
  __syncthreads();
  doublex4 acc[NRB][NCB];
#pragma unroll
  for (int a = 0; a < NRB; ++a)
#pragma unroll
    for (int b = 0; b < NCB; ++b) acc[a][b] = doublex4{0.0, 0.0, 0.0, 0.0};
  auto io = momentum_io<RP, NRB, NCB>(Xin, Vin, r0, rows, q, l16, [](int a) { return 16 * a; },
                                      [=](int b) { return 16 * (wave + 4 * b); });
  const double* gcol = Gneg + 16 * wave + l16;  // column block b of this wave: + 64 b
  double pre[PD][NCB];
#pragma unroll
  for (int d = 0; d < PD; ++d)
#pragma unroll
    for (int b = 0; b < NCB; ++b) pre[d][b] = gcol[(int64_t)(4 * d + q) * RP + 64 * b];
  for (int k0 = 0; k0 < RP; k0 += 4 * PD) {
#pragma unroll
    for (int d = 0; d < PD; ++d) {
      const int k = k0 + 4 * d;
      double bv[NCB];
#pragma unroll
      for (int b = 0; b < NCB; ++b) bv[b] = pre[d][b];
      const int kn = k + 4 * PD;
      if (kn < RP) {
#pragma unroll
        for (int b = 0; b < NCB; ++b) pre[d][b] = gcol[(int64_t)(kn + q) * RP + 64 * b];
      }
#pragma unroll
      for (int a = 0; a < NRB; ++a) {
        const double av = (double)ys[(16 * a + l16) * LS + k + q];
#pragma unroll
        for (int b = 0; b < NCB; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f64_16x16x4f64(av, bv[b], acc[a][b], 0, 0, 0);
      }
    }
  }
  const bool bad = io.finish(acc, Xout, Vout, eta, gamma);
  if (bad) flag_status(status, STATUS_NONFINITE, step_id);
}

hipError_t launch_apply(const float* Ypart, int64_t y_stride, int nsplit, const float* Ysp,
                        const double* Gneg,
                        const float* Xin, const float* Vin, float* Xout, float* Vout,
                        int64_t rows, int rp, float eta, float gamma, int* status, int step_id,
                        hipStream_t st) {
  if (rows <= 0) return hipSuccess;
#define CASE(R)                                                                              \
  case R: {                                                                                  \
    constexpr int RW = ApplyCfg<R>::RW;                                                      \
    hipLaunchKernelGGL((apply_kernel<R>), dim3((unsigned)((rows + RW - 1) / RW)), dim3(256), 0, \
                       st, Ypart, y_stride, nsplit, Ysp, Gneg, Xin, Vin, Xout, Vout, rows, eta,   \
                       gamma, status, step_id);                                              \
    break;                                                                                   \
  }
  // Row tile: the tallest allowed one that still gives 4096 workgroups (1024 at r_p >= 512),
  // else 16 rows.  Every workgroup reads all of G^-1 (r_p^2 doubles) from L2 once, so at
  // r_p = 512 a 16-row tile moves 128 KB of it per row, which saturates the L2; 32 rows halve
  // that at fewer workgroups.
  const int rw_max = rp >= 64 ? (16384 / rp >= 64 ? 64 : (16384 / rp >= 32 ? 32 : 16)) : 16;
  const int64_t min_wgs = rp >= 512 ? 1024 : 4096;
  int rw = 16;
  for (int cand = rw_max; cand > 16; cand /= 2)
    if ((rows + cand - 1) / cand >= min_wgs) {
      rw = cand;
      break;
    }
#define WIDE_RW(R, W)                                                                        \
  hipLaunchKernelGGL((apply_wide_kernel<R, W>), dim3((unsigned)((rows + W - 1) / W)), dim3(256), \
                     0, st, Ypart, y_stride, nsplit, Ysp, Gneg, Xin, Vin, Xout, Vout, rows, eta,  \
                     gamma, status, step_id)
#define WIDE(R)                                                                              \
  case R: {                                                                                  \
    if (rw >= 64 && wide_max_rw<R>() >= 64) WIDE_RW(R, (wide_max_rw<R>() >= 64 ? 64 : 16)); \
    else if (rw >= 32 && wide_max_rw<R>() >= 32) WIDE_RW(R, (wide_max_rw<R>() >= 32 ? 32 : 16)); \
    else WIDE_RW(R, 16);                                                                     \
    break;                                                                                   \
  }
  switch (rp) {
    CASE(16) CASE(32) CASE(48)
    WIDE(64) WIDE(128) WIDE(192) WIDE(256) WIDE(320) WIDE(384) WIDE(448) WIDE(512)
    default: return hipErrorInvalidValue;
  }
#undef CASE
#undef WIDE
#undef WIDE_RW
  return hipGetLastError();
}

}  // namespace nmd
