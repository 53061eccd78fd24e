// Fused dense contraction Y = min(0, X P^T) P on gfx950 fp32 MFMA.
//
// This is the dense part of Z_{:,J} P_J (eq. updateZ contracted as in eqs. lsqA / lsqA_sto):
// on the zeros of S the auxiliary matrix equals min(0, L); the sparse correction adds the
// nonzeros afterwards.  The L tile is produced by MFMA, clamped in registers and consumed by
// MFMA; neither L nor Z reaches memory (the IO-aware fusion of Sec. 4.2, with the clamp-then-
// contract order and the raw panel P instead of a pseudo-inverse).
//
// Layout and data flow (one workgroup = 4 waves, one per SIMD):
//   * X: rows x RP row-major (RP = padded rank, zero columns beyond r).  Each wave keeps
//     16*MI rows of X resident in VGPRs as MFMA operands for the whole launch.
//   * P rows of the split's column range stream through LDS in tiles of NT rows (row stride
//     RP+4 floats, which keeps both read patterns below free of bank conflicts).
//   * GEMM1 computes the TRANSPOSED tile L^T (16 j x 16 i) with v_mfma_f32_16x16x4f32:
//     srcA = P fragment (row j = lane%16), srcB = X fragment (row i = lane%16), both over the
//     same permuted k order (lane group q = lane/16 holds k = 16t + 4q + c, c = 0..3, so one
//     ds_read_b128 serves four k-steps).  The accumulator of lane l, register v then holds
//     L[i = l%16][j = 4q + v], which is exactly the srcA layout GEMM2 needs for the k-slice
//     {4q + v}: the clamped tile feeds GEMM2 without any data movement.
//   * GEMM2: Y[i][c] += sum_j min(0, L[i][j]) P[j][c], srcB read from LDS as single floats.
//   * Split-J: the workgroups of one row tile are spread over `nsplit` disjoint ranges of P
//     rows, each writing its own partial Y; the solve kernel sums them in fp64.  Short fp32
//     accumulation chains keep the rounding error of Y small, which matters because the Gram
//     solve amplifies it by the condition number of P^T P.
//   * blockIdx is remapped so that each XCD (dispatch round-robins workgroups over the 8 XCDs)
//     receives a contiguous run of (split, row tile) pairs, so a split's P range stays in the
//     L2 of one or two XCDs.

#include "nmd_internal.h"

namespace nmd {

typedef float floatx4 __attribute__((ext_vector_type(4)));

template <int RP>
struct DenseCfg;
// MI: 16-row blocks of X per wave (4 waves per workgroup).  NT: P rows per LDS tile.
template <> struct DenseCfg<16>  { static constexpr int MI = 4, NT = 512; };
template <> struct DenseCfg<32>  { static constexpr int MI = 4, NT = 256; };
template <> struct DenseCfg<48>  { static constexpr int MI = 4, NT = 160; };
template <> struct DenseCfg<64>  { static constexpr int MI = 4, NT = 128; };
template <> struct DenseCfg<128> { static constexpr int MI = 4, NT = 64; };
template <> struct DenseCfg<192> { static constexpr int MI = 2, NT = 32; };
template <> struct DenseCfg<256> { static constexpr int MI = 2, NT = 32; };
template <> struct DenseCfg<320> { static constexpr int MI = 1, NT = 16; };
template <> struct DenseCfg<384> { static constexpr int MI = 1, NT = 16; };
template <> struct DenseCfg<448> { static constexpr int MI = 1, NT = 16; };
template <> struct DenseCfg<512> { static constexpr int MI = 1, NT = 16; };

int padded_rank(int r) {
  if (r <= 64) return ((r + 15) / 16) * 16;
  return ((r + 63) / 64) * 64;
}

template <int RP>
static constexpr int rows_per_wg() { return 64 * DenseCfg<RP>::MI; }

int dense_rows_per_wg(int rp) {
  switch (rp) {
    case 16: return rows_per_wg<16>();
    case 32: return rows_per_wg<32>();
    case 48: return rows_per_wg<48>();
    case 64: return rows_per_wg<64>();
    case 128: return rows_per_wg<128>();
    case 192: return rows_per_wg<192>();
    case 256: return rows_per_wg<256>();
    case 320: return rows_per_wg<320>();
    case 384: return rows_per_wg<384>();
    case 448: return rows_per_wg<448>();
    case 512: return rows_per_wg<512>();
  }
  return 0;
}

// Logical workgroup index so that XCD x (= blockIdx % 8) owns a contiguous range.
__device__ __forceinline__ int64_t xcd_logical(int64_t bid, int64_t total) {
  const int64_t x = bid & 7, local = bid >> 3;
  const int64_t per = total >> 3, rem = total & 7;
  return x * per + (x < rem ? x : rem) + local;
}

// OBJ = false: Y partial outputs.  OBJ = true: per-workgroup fp64 sum of max(0, L)^2.
template <int RP, bool OBJ>
__global__ __launch_bounds__(256, 1) void dense_kernel(
    const float* __restrict__ X, int64_t rows, const float* __restrict__ P, int64_t blk,
    float* __restrict__ Ypart, int64_t y_stride, int nsplit, int64_t row_tiles,
    double* __restrict__ partial) {
  constexpr int MI = DenseCfg<RP>::MI;
  constexpr int NT = DenseCfg<RP>::NT;
  constexpr int KS = RP / 4;    // k-steps of GEMM1
  constexpr int KG = RP / 16;   // groups of four k-steps (one ds_read_b128 each)
  constexpr int CB = RP / 16;   // 16-column blocks of Y
  constexpr int LS = RP + 4;    // LDS row stride (floats)
  constexpr int NV4 = NT * RP / 4;            // float4 per tile
  constexpr int NLD = (NV4 + 255) / 256;      // float4 loads per thread per tile
  __shared__ __attribute__((aligned(16))) float tile[NT * LS];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int q = lane >> 4, l16 = lane & 15;

  const int64_t logical = xcd_logical(blockIdx.x, (int64_t)gridDim.x);
  const int split = (int)(logical / row_tiles);
  const int64_t rt = logical - (int64_t)split * row_tiles;
  const int64_t jb0 = (int64_t)split * blk / nsplit;
  const int64_t jb1 = (int64_t)(split + 1) * blk / nsplit;
  const int64_t row0 = rt * (64 * MI) + (int64_t)wave * (16 * MI);

  // Resident X fragments: a[mi][4t + c] = X[row0 + 16 mi + l16][16t + 4q + c].
  float a[MI][KS];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
    const int64_t row = row0 + 16 * mi + l16;
#pragma unroll
    for (int t = 0; t < KG; ++t) {
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (row < rows) v = *reinterpret_cast<const float4*>(X + row * RP + 16 * t + 4 * q);
      a[mi][4 * t + 0] = v.x;
      a[mi][4 * t + 1] = v.y;
      a[mi][4 * t + 2] = v.z;
      a[mi][4 * t + 3] = v.w;
    }
  }

  floatx4 y[OBJ ? 1 : MI][OBJ ? 1 : CB];
  if constexpr (!OBJ) {
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) y[mi][cb] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  double objsum = 0.0;

  // Prefetch registers for the next tile.
  float4 pf[NLD];
  auto fetch = [&](int64_t j0) {
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int f = tid + 256 * u;
      const int rr = f / (RP / 4), c4 = f - rr * (RP / 4);
      const int64_t j = j0 + rr;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (f < NV4 && j < jb1) v = *reinterpret_cast<const float4*>(P + j * RP + 4 * c4);
      pf[u] = v;
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int f = tid + 256 * u;
      const int rr = f / (RP / 4), c4 = f - rr * (RP / 4);
      if (f < NV4) *reinterpret_cast<float4*>(&tile[rr * LS + 4 * c4]) = pf[u];
    }
  };

  if (jb0 < jb1) fetch(jb0);
  for (int64_t j0 = jb0; j0 < jb1; j0 += NT) {
    __syncthreads();  // previous tile fully consumed
    stash();
    __syncthreads();
    if (j0 + NT < jb1) fetch(j0 + NT);
    const int njb = (int)((jb1 - j0 + 15) / 16) < NT / 16 ? (int)((jb1 - j0 + 15) / 16) : NT / 16;
    for (int jb = 0; jb < njb; ++jb) {
      floatx4 lt[MI];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) lt[mi] = floatx4{0.f, 0.f, 0.f, 0.f};
      const float* brow = &tile[(jb * 16 + l16) * LS + 4 * q];
#pragma unroll
      for (int t = 0; t < KG; ++t) {
        const float4 bv = *reinterpret_cast<const float4*>(brow + 16 * t);
#pragma unroll
        for (int mi = 0; mi < MI; ++mi) {
          lt[mi] = __builtin_amdgcn_mfma_f32_16x16x4f32(bv.x, a[mi][4 * t + 0], lt[mi], 0, 0, 0);
          lt[mi] = __builtin_amdgcn_mfma_f32_16x16x4f32(bv.y, a[mi][4 * t + 1], lt[mi], 0, 0, 0);
          lt[mi] = __builtin_amdgcn_mfma_f32_16x16x4f32(bv.z, a[mi][4 * t + 2], lt[mi], 0, 0, 0);
          lt[mi] = __builtin_amdgcn_mfma_f32_16x16x4f32(bv.w, a[mi][4 * t + 3], lt[mi], 0, 0, 0);
        }
      }
      if constexpr (OBJ) {
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const float p = fmaxf(lt[mi][v], 0.f);
            objsum += (double)(p * p);
          }
      } else {
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
          for (int v = 0; v < 4; ++v) lt[mi][v] = fminf(lt[mi][v], 0.f);
        const float* b2 = &tile[(jb * 16 + 4 * q) * LS + l16];
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const float bb = b2[v * LS + 16 * cb];
#pragma unroll
            for (int mi = 0; mi < MI; ++mi)
              y[mi][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(lt[mi][v], bb, y[mi][cb], 0, 0, 0);
          }
        }
      }
    }
  }

  if constexpr (OBJ) {
    // workgroup reduction in a fixed order
    __shared__ double red[256];
    red[tid] = objsum;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
      if (tid < s) red[tid] += red[tid + s];
      __syncthreads();
    }
    if (tid == 0) partial[logical] = red[0];
  } else {
    float* Y = Ypart + (int64_t)split * y_stride;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t row = row0 + 16 * mi + 4 * q + v;
        if (row < rows) {
#pragma unroll
          for (int cb = 0; cb < CB; ++cb) Y[row * RP + 16 * cb + l16] = y[mi][cb][v];
        }
      }
  }
}

template <int RP, bool OBJ>
static hipError_t launch_dense_t(const float* X, int64_t rows, const float* P, int64_t blk,
                                 float* Ypart, int64_t y_stride, int nsplit, double* partial,
                                 hipStream_t st) {
  const int64_t row_tiles = (rows + rows_per_wg<RP>() - 1) / rows_per_wg<RP>();
  const int64_t total = row_tiles * nsplit;
  if (total <= 0) return hipSuccess;
  if (total > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL((dense_kernel<RP, OBJ>), dim3((unsigned)total), dim3(256), 0, st, X, rows, P,
                     blk, Ypart, y_stride, nsplit, row_tiles, partial);
  return hipGetLastError();
}

#define NMD_RP_DISPATCH(rp, CALL) \
  switch (rp) {                   \
    case 16: return CALL(16);     \
    case 32: return CALL(32);     \
    case 48: return CALL(48);     \
    case 64: return CALL(64);     \
    case 128: return CALL(128);   \
    case 192: return CALL(192);   \
    case 256: return CALL(256);   \
    case 320: return CALL(320);   \
    case 384: return CALL(384);   \
    case 448: return CALL(448);   \
    case 512: return CALL(512);   \
  }                               \
  return hipErrorInvalidValue;

hipError_t launch_dense(const float* X, int64_t rows, const float* P, int64_t blk, int rp,
                        float* Ypart, int64_t y_stride, int nsplit, hipStream_t st) {
#define CALL(R) launch_dense_t<R, false>(X, rows, P, blk, Ypart, y_stride, nsplit, nullptr, st)
  NMD_RP_DISPATCH(rp, CALL)
#undef CALL
}

int dense_max_wgs(int64_t rows, int rp, int nsplit) {
  const int rw = dense_rows_per_wg(rp);
  return rw ? (int)(((rows + rw - 1) / rw) * nsplit) : 0;
}

hipError_t launch_obj_dense(const float* X, int64_t rows, const float* P, int64_t cols, int rp,
                            double* partial, int* npartial, hipStream_t st) {
  // Enough column splits to give the GPU a few thousand workgroups.
  const int rw = dense_rows_per_wg(rp);
  if (!rw) return hipErrorInvalidValue;
  const int64_t row_tiles = (rows + rw - 1) / rw;
  int64_t ns = (2048 + row_tiles - 1) / row_tiles;
  if (ns > 64) ns = 64;
  if (ns > cols) ns = cols;
  if (ns < 1) ns = 1;
  *npartial = (int)(row_tiles * ns);
  const int nsplit = (int)ns;
#define CALL(R) launch_dense_t<R, true>(X, rows, P, cols, nullptr, 0, nsplit, partial, st)
  NMD_RP_DISPATCH(rp, CALL)
#undef CALL
}

}  // namespace nmd
