// Fused dense contraction Y = sgn * max(0, X P^T) P on gfx950 fp32 MFMA (kernel templates; the
// instantiations live in dense.hip for r_p <= 256 and in dense_large.hip for larger ranks, which
// are compiled with different register-allocation flags).
//
// With L = X P_J^T and S-hat = max(0, L) (eq. rectify), the difference matrix of eq. updateD
// gives Delta_{:J} P_J = sum over the nonzeros of S of (S - min(0, L)) p_j  -  S-hat P_J, and
// the least-squares update is X <- X + Delta_{:J} P_J (P_J^T P_J)^-1 (eqs. spLsqA, lsqA_sto).
// This kernel forms the dense term -S-hat P_J (sgn = -1); the sparse correction adds the first
// term.  S-hat is mostly zero (the factors start with opposite signs and the fit keeps it sparse,
// Sec. 4.3), so a wave skips the MFMAs of every 16 x 4 operand slice of S-hat that holds no
// positive entry, and (at r_p = 256 and 512) runs the second product per 4-row quad-column of
// S-hat on 4 x 4 x 1 MFMAs, only where one holds a positive entry (below).  The L tile is produced by
// MFMA, rectified in registers and consumed by MFMA; neither L nor S-hat reaches memory (the
// IO-aware fusion of Sec. 4.2, with the raw panel P instead of a pseudo-inverse).
//
// Data flow (one workgroup = WAVES waves: 8 at r_p = 128 and 256, two per SIMD; 4 elsewhere):
//   * X: rows x RP row-major (RP = padded rank, zero columns beyond r).  Each wave keeps
//     16*MI rows of X resident in VGPRs as MFMA operands for the whole launch.
//   * P rows of the split's range stream through LDS (row stride RP + 4 floats, which keeps
//     both read patterns free of bank conflicts); the next tile is in flight while the current
//     one is consumed.
//   * GEMM1 builds the transposed tile L^T (16 j x 16 i); the accumulator of lane l, register
//     v holds L[i = l%16][j = 4(l/16) + v], which is exactly the srcA layout of GEMM2 for the
//     k-slice {4(l/16) + v}: the rectified tile feeds GEMM2 with no data movement.
//   * GEMM2: Y[i][c] += sum_j max(0, L[i][j]) P[j][c], srcB read from LDS, per 16 x 4 slice
//     of max(0, L) on 16 x 16 x 4 MFMAs, skipped when zero; at r_p = 256 and 512 per
//     quad-column (4 rows x 1 column) on 4 x 4 x 1 MFMAs with the A operand broadcast from
//     the L tile.
//   * Split-J: the workgroups of one row tile may be spread over `nsplit` disjoint ranges of P
//     rows, each writing its own partial Y; the solve kernel sums them in fp64.

#pragma once

#include "tile.h"

namespace nmd {

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) void glb_void;

// Launch shape per padded rank.  MI: 16-row blocks of X per wave; WAVES: waves per workgroup
// (8 puts two waves on each SIMD, so that one wave's MFMAs cover the other's LDS waits,
// accumulator read-outs and branches); NT: panel rows per LDS tile; RING: slices of the second
// product whose operands are read during the first (4: all of them, where registers allow);
// DIRECT: direct global->LDS loads into double-buffered tiles (for long rows; register staging
// there pushes the VGPR budget into spills) instead of register staging through one tile (a
// direct load moves 64 chunks of one row, so short rows would leave most lanes idle); QUAD:
// the second product runs per quad-column (below) and no operand ring is kept (RING unused).
template <int RP>
struct DenseLaunch {
  static constexpr int MI = DenseCfg<RP>::MI;
  static constexpr int WAVES = 4;
  static constexpr bool DIRECT = RP >= 320;
  static constexpr int NT = DIRECT ? DenseCfg<RP>::NTD : DenseCfg<RP>::NT;
  static constexpr int RING = RP >= 320 ? 4 : 2;
  static constexpr bool QUAD = RP == 512;
};
template <>
struct DenseLaunch<256> {
  static constexpr int MI = 1;
  static constexpr int WAVES = 8;
  static constexpr bool DIRECT = true;
  static constexpr int NT = 64;
  static constexpr int RING = 4;
  static constexpr bool QUAD = true;
};
template <>
struct DenseLaunch<128> {
  static constexpr int MI = 2;
  static constexpr int WAVES = 8;
  static constexpr bool DIRECT = true;
  static constexpr int NT = 128;
  static constexpr int RING = 4;
  static constexpr bool QUAD = false;
};

template <int RP>
constexpr int dense_rows() { return 16 * DenseLaunch<RP>::MI * DenseLaunch<RP>::WAVES; }

// Direct staging of panel rows j0 .. j0+NT-1 from global memory straight into a padded LDS
// tile; wave w fills rows w, w + WAVES, ...; a direct load writes 64 consecutive 16-byte chunks
// (lane l -> chunk l), so each instruction covers up to 64 chunks of one row.  Rows past the
// split end are zero-filled with ordinary LDS stores (their L is then zero).
template <int RP>
__device__ __forceinline__ void issue_tile(float* dst, const float* __restrict__ P, int64_t j0,
                                           int64_t jb1, int wave, int lane) {
  constexpr int WAVES = DenseLaunch<RP>::WAVES;
  constexpr int NT = DenseLaunch<RP>::NT;
  constexpr int LS = RP + 4;
  constexpr int CPR = RP / 4;
  constexpr int IPR = (CPR + 63) / 64;
#pragma unroll
  for (int rr = 0; rr < NT / WAVES; ++rr) {
    const int r = wave + WAVES * rr;
    const int64_t jr = j0 + r;
    if (jr < jb1) {
      const float* src = P + jr * RP;
#pragma unroll
      for (int k = 0; k < IPR; ++k) {
        const int c = 64 * k + lane;
        if (CPR % 64 == 0 || c < CPR)
          __builtin_amdgcn_global_load_lds((glb_void*)(src + 4 * c),
                                           (lds_void*)(dst + r * LS + 256 * k), 16, 0, 0);
      }
    } else {
#pragma unroll
      for (int k = 0; k < IPR; ++k) {
        const int c = 64 * k + lane;
        if (CPR % 64 == 0 || c < CPR)
          *reinterpret_cast<float4*>(dst + r * LS + 4 * c) = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
  }
}

// Second product by quad-columns on v_mfma_f32_4x4x1f32 (16 blocks of 4 x 4 x 1 each).  A
// quad-column is 4 rows (4 q4 .. 4 q4 + 3) of one column j of the rectified tile z; it sits in
// register v = j % 4 of lanes 16 (j / 4) + 4 q4 + 0..3, i.e. in block n = 4 (j / 4) + q4 of the
// instruction's A operand.  With the broadcast controls set so that all 16 blocks take the A
// operand of block n (CBSZ = 4, ABID = n), one instruction adds z[4 q4 + 0..3][j] P[j][c] for
// 64 columns c: block b, column c' of the output is lane 4 b + c' of the B operand, which holds
// P[j][G lane + g].  So G = RP / 64 instructions cover a quad-column, with no data movement
// between lanes.  Only quad-columns holding a positive entry run (wave ballots).  An isolated
// positive entry costs G instructions of 8 cycles; a fully positive 16 x 4 slice (16
// quad-columns) costs the same matrix-core time as its 16 x 16 x 4 form.
// Accumulator y[G q4 + g], register v, lane l holds Y[4 q4 + v][G l + g].
// Returns the number of positive entries of the block.
template <int RP, int V, int QQ, int Q4>
__device__ __forceinline__ void quad_mfma(floatx4 (&y)[RP / 16], const floatx4& z,
                                          const float (&bb)[RP / 64]) {
  constexpr int G = RP / 64;
#pragma unroll
  for (int g = 0; g < G; ++g)
    y[G * Q4 + g] = __builtin_amdgcn_mfma_f32_4x4x1f32(z[V], bb[g], y[G * Q4 + g], 4, 4 * QQ + Q4, 0);
}

template <int RP, int V, int QQ>
__device__ __forceinline__ unsigned quad_group(floatx4 (&y)[RP / 16], const floatx4& z,
                                               unsigned b16, const float* tile, int jb, int lane) {
  constexpr int G = RP / 64;
  const float* prow = &tile[(jb * 16 + 4 * QQ + V) * (RP + 4) + G * lane];
  float bb[G];
#pragma unroll
  for (int h = 0; h < G / 4; ++h) {
    const float4 t = *reinterpret_cast<const float4*>(prow + 4 * h);
    bb[4 * h + 0] = t.x;
    bb[4 * h + 1] = t.y;
    bb[4 * h + 2] = t.z;
    bb[4 * h + 3] = t.w;
  }
  unsigned cnt = 0;
  if (b16 & 0x000fu) { cnt += __builtin_popcount(b16 & 0x000fu); quad_mfma<RP, V, QQ, 0>(y, z, bb); }
  if (b16 & 0x00f0u) { cnt += __builtin_popcount(b16 & 0x00f0u); quad_mfma<RP, V, QQ, 1>(y, z, bb); }
  if (b16 & 0x0f00u) { cnt += __builtin_popcount(b16 & 0x0f00u); quad_mfma<RP, V, QQ, 2>(y, z, bb); }
  if (b16 & 0xf000u) { cnt += __builtin_popcount(b16 & 0xf000u); quad_mfma<RP, V, QQ, 3>(y, z, bb); }
  return cnt;
}

template <int RP, int V>
__device__ __forceinline__ unsigned quad_slice(floatx4 (&y)[RP / 16], const floatx4& z,
                                               const float* tile, int jb, int lane) {
  const unsigned long long bits = __ballot(z[V] > 0.f);
  if (!bits) return 0;
  unsigned cnt = 0;
  const unsigned lo = (unsigned)bits, hi = (unsigned)(bits >> 32);
  if (lo & 0xffffu) cnt += quad_group<RP, V, 0>(y, z, lo & 0xffffu, tile, jb, lane);
  if (lo >> 16) cnt += quad_group<RP, V, 1>(y, z, lo >> 16, tile, jb, lane);
  if (hi & 0xffffu) cnt += quad_group<RP, V, 2>(y, z, hi & 0xffffu, tile, jb, lane);
  if (hi >> 16) cnt += quad_group<RP, V, 3>(y, z, hi >> 16, tile, jb, lane);
  return cnt;
}

template <int RP>
__device__ __forceinline__ unsigned quad_block(floatx4 (&y)[RP / 16], const floatx4& z,
                                               const float* tile, int jb, int lane) {
  static_assert(RP == 256 || RP == 512, "quad-column path: r_p = 256 or 512");
  return quad_slice<RP, 0>(y, z, tile, jb, lane) + quad_slice<RP, 1>(y, z, tile, jb, lane) +
         quad_slice<RP, 2>(y, z, tile, jb, lane) + quad_slice<RP, 3>(y, z, tile, jb, lane);
}

// Both products over the panel rows j0 .. min(j0 + NT, jb1) - 1 held in the LDS tile; returns
// the number of 16 x 4 slices of max(0, L) that ran the second product whole, and adds the
// positive entries taken by quad-columns to `entries`.
template <int RP>
__device__ __forceinline__ unsigned consume_tile(const float* tile, int64_t j0, int64_t jb1,
                                                 const float (&a)[DenseLaunch<RP>::MI][RP / 4],
                                                 floatx4 (&y)[DenseLaunch<RP>::MI][RP / 16],
                                                 int q, int l16, unsigned& entries) {
  constexpr int MI = DenseLaunch<RP>::MI;
  constexpr int NT = DenseLaunch<RP>::NT;
  constexpr int CB = RP / 16;
  const int left = (int)((jb1 - j0 + 15) / 16);
  const int njb = left < NT / 16 ? left : NT / 16;
  unsigned done = 0;
  float4 pre[l_lookahead<RP>()];
  l_prefetch<RP>(pre, tile, 0, q, l16);
  if constexpr (DenseLaunch<RP>::QUAD) {
    static_assert(MI == 1, "quad-column second product: one 16-row block per wave");
    // Every j-block of the tile runs (rows past the split end are zero in LDS, so their L is
    // zero and they add nothing).  A block's second product runs after the next block's first
    // product has been issued, from the accumulator chains held meanwhile, so that the wave
    // does not wait for its first product to drain before the branches of the second.
    static_assert(l_chains<1>() == 2, "two accumulator chains");
    floatx4 hold[2];
#pragma unroll
    for (int jb = 0; jb < NT / 16; ++jb) {
      float ring[1][CB];
      floatx4 acc[2][1];
      l_tile_acc<RP, 1, 0>(acc, a, pre, ring, tile, jb, q, l16);
      if (jb + 1 < NT / 16) l_prefetch<RP>(pre, tile, jb + 1, q, l16);
      if (jb > 0) {
        floatx4 z = hold[0] + hold[1];
#pragma unroll
        for (int v = 0; v < 4; ++v) z[v] = z[v] > 0.f ? z[v] : 0.f;
        entries += quad_block<RP>(y[0], z, tile, jb - 1, q * 16 + l16);
      }
      hold[0] = acc[0][0];
      hold[1] = acc[1][0];
    }
    floatx4 z = hold[0] + hold[1];
#pragma unroll
    for (int v = 0; v < 4; ++v) z[v] = z[v] > 0.f ? z[v] : 0.f;
    entries += quad_block<RP>(y[0], z, tile, NT / 16 - 1, q * 16 + l16);
    (void)njb;
  } else {
    constexpr int NR = DenseLaunch<RP>::RING;
    for (int jb = 0; jb < njb; ++jb) {
      // the block's second-product operands are read inside its first product
      float ring[NR][CB];
      floatx4 lt[MI];
      l_tile<RP, MI, NR>(lt, a, pre, ring, tile, jb, q, l16);
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int v = 0; v < 4; ++v) lt[mi][v] = lt[mi][v] > 0.f ? lt[mi][v] : 0.f;
      const unsigned live = live_slices<MI>(lt);
      // the next block's first panel fragments, in flight during this block's second product
      if (jb + 1 < njb) l_prefetch<RP>(pre, tile, jb + 1, q, l16);
      done += zb_tile<RP, MI, NR>(y, lt, live, ring, tile, jb, q, l16);
    }
  }
  return done;
}

// One step of the double-buffered direct pipeline: start the loads of the next tile into `nxt`
// (when not null) and consume the current tile `cur`.  The two are distinct LDS buffers; the
// restrict qualifiers tell the compiler that the reads of `cur` do not depend on the direct
// loads into `nxt`, so it need not wait for those loads before the products start.
template <int RP>
__device__ __forceinline__ unsigned direct_step(
    const float* __restrict__ cur, float* __restrict__ nxt, const float* __restrict__ P,
    int64_t j0, int64_t jb1, const float (&a)[DenseLaunch<RP>::MI][RP / 4],
    floatx4 (&y)[DenseLaunch<RP>::MI][RP / 16], int wave, int lane, int q, int l16,
    unsigned& entries) {
  if (nxt) issue_tile<RP>(nxt, P, j0 + DenseLaunch<RP>::NT, jb1, wave, lane);
  return consume_tile<RP>(cur, j0, jb1, a, y, q, l16, entries);
}

template <int RP>
__global__ __launch_bounds__(64 * DenseLaunch<RP>::WAVES) void dense_kernel(
    const float* __restrict__ X, int64_t rows, const float* __restrict__ P, int64_t blk,
    float* __restrict__ Ypart, int64_t y_stride, int nsplit, int64_t row_tiles, float sgn,
    unsigned long long* __restrict__ gemm2_blocks) {
  constexpr int MI = DenseLaunch<RP>::MI;
  constexpr int WAVES = DenseLaunch<RP>::WAVES;
  constexpr int CB = RP / 16;
  constexpr int LS = RP + 4;  // padded LDS row stride (floats)
  constexpr bool DIRECT = DenseLaunch<RP>::DIRECT;
  constexpr int NT = DenseLaunch<RP>::NT;
  static_assert(NT % 16 == 0 && NT % WAVES == 0, "tile shape");
  __shared__ __attribute__((aligned(16))) float smem[(DIRECT ? 2 : 1) * NT * LS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q = lane >> 4, l16 = lane & 15;

  const int64_t logical = xcd_logical(blockIdx.x, (int64_t)gridDim.x);
  const int split = (int)(logical / row_tiles);
  const int64_t rt = logical - (int64_t)split * row_tiles;
  const int64_t jb0 = (int64_t)split * blk / nsplit;
  const int64_t jb1 = (int64_t)(split + 1) * blk / nsplit;
  const int64_t row0 = rt * dense_rows<RP>() + (int64_t)wave * (16 * MI);

  float a[MI][RP / 4];
  load_x_frags<RP, MI>(a, X, rows, row0, q, l16);

  floatx4 y[MI][CB];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) y[mi][cb] = floatx4{0.f, 0.f, 0.f, 0.f};

  unsigned int done = 0;     // 16 x 4 slices of max(0, L) whose second product ran whole
  unsigned int entries = 0;  // positive entries of max(0, L) taken by quad-columns

  if constexpr (DIRECT) {
    if (jb0 < jb1) issue_tile<RP>(smem, P, jb0, jb1, wave, lane);
    int cur = 0;
    for (int64_t j0 = jb0; j0 < jb1; j0 += NT, cur ^= 1) {
      __builtin_amdgcn_s_waitcnt(0);  // this wave's loads of the tile have landed
      __syncthreads();                // every wave's have; the other buffer is free again
      done += direct_step<RP>(smem + cur * (NT * LS), j0 + NT < jb1 ? smem + (cur ^ 1) * (NT * LS) : nullptr,
                              P, j0, jb1, a, y, wave, lane, q, l16, entries);
    }
  } else {
    // register staging: the next tile's global loads are in flight while this one is consumed
    // (rows past the split end are stored as zeros)
    PanelTile<RP, NT, 64 * WAVES> pt;
    if (jb0 < jb1) pt.fetch(P, jb0, jb1, tid);
    for (int64_t j0 = jb0; j0 < jb1; j0 += NT) {
      __syncthreads();  // previous tile fully consumed
      pt.stash(smem, tid);
      __syncthreads();
      if (j0 + NT < jb1) pt.fetch(P, j0 + NT, jb1, tid);
      done += consume_tile<RP>(smem, j0, jb1, a, y, q, l16, entries);
    }
  }

  float* Y = Ypart + (int64_t)split * y_stride;
  if constexpr (DenseLaunch<RP>::QUAD) {
    // quad-column layout: y[G q4 + g], lane l, register v holds Y[row0 + 4 q4 + v][G l + g]
    constexpr int G = RP / 64;
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t row = row0 + 4 * q4 + v;
        if (row < rows) {
#pragma unroll
          for (int h = 0; h < G / 4; ++h)
            *reinterpret_cast<float4*>(&Y[row * RP + G * lane + 4 * h]) =
                make_float4(sgn * y[0][G * q4 + 4 * h + 0][v], sgn * y[0][G * q4 + 4 * h + 1][v],
                            sgn * y[0][G * q4 + 4 * h + 2][v], sgn * y[0][G * q4 + 4 * h + 3][v]);
        }
      }
  } else {
  // Y block (16 x 16): lane l, register v holds Y[row0 + 16 mi + 4q + v][16 cb + l16].
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t row = row0 + 16 * mi + 4 * q + v;
      if (row < rows) {
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) Y[row * RP + 16 * cb + l16] = sgn * y[mi][cb][v];
      }
    }
  }
  if (gemm2_blocks && lane == 0) {
    atomicAdd(gemm2_blocks, (unsigned long long)done);
    if (entries) atomicAdd(gemm2_blocks + 1, (unsigned long long)entries);
  }
}

template <int RP>
static hipError_t launch_dense_t(const float* X, int64_t rows, const float* P, int64_t blk,
                                 float* Ypart, int64_t y_stride, int nsplit, float sgn,
                                 unsigned long long* gemm2_blocks, hipStream_t st) {
  const int64_t row_tiles = (rows + dense_rows<RP>() - 1) / dense_rows<RP>();
  const int64_t total = row_tiles * nsplit;
  if (total <= 0) return hipSuccess;
  if (total > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL((dense_kernel<RP>), dim3((unsigned)total),
                     dim3(64 * DenseLaunch<RP>::WAVES), 0, st, X, rows, P, blk,
                     Ypart, y_stride, nsplit, row_tiles, sgn, gemm2_blocks);
  return hipGetLastError();
}

template <int RP>
static hipError_t wgs_per_cu_t(int* out) {
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(out, dense_kernel<RP>,
                                                      64 * DenseLaunch<RP>::WAVES, 0);
}

}  // namespace nmd
