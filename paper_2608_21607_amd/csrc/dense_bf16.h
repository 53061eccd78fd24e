// Rectified contraction Y = sgn * max(0, X P^T) P with both products on bf16 MFMA of two-term
// operand splits (x = x_hi + x_lo, x_hi = bf16(x), x_lo = bf16(x - x_hi): 16 significant bits),
// for a dense max(0, L): the gfx950 counterpart of the paper's TF32 fused kernels (Sec. 4.2) at
// their kernel-throughput shape.  Each product is three bf16 products (hi hi, hi lo, lo hi)
// accumulated in fp32; the dropped lo lo terms and the split remainders are about 2^-16 of
// sum |a_k b_k| per output.
//
// This header holds the helpers of both forms and the 32 x 32 x 16 form (padded ranks 16 to
// 128); the 16 x 16 x 32 form (256 and 512) is in dense_bf16_large.hip.  In the 16 x 16 form a
// wave holds 16 rows of X and takes the panel 32 rows at a time: its first product gives lane
// (q, l16), register v, L[i = l16][j = 4q + v] and L[i = l16][j = 16 + 4q + v]; those eight
// values, rectified and split (zsplit), are the srcA operand of one K = 32 MFMA of the second
// product, A[i = l16][k = 8q + e] with k <-> panel row 4q + e (e < 4), 16 + 4q + e - 4 (e >= 4).

#pragma once

#include "dense_kernel.h"

namespace nmd {
namespace bx {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) unsigned u32x4;

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(2))) float floatx2;

// Two values rounded to bf16 (nearest even), packed: element 0 in the low half.
__device__ __forceinline__ unsigned bf16_pair(floatx2 x) {
  return __builtin_bit_cast(unsigned, __builtin_convertvector(x, bf16x2));
}

// Eight values as packed hi and lo operands (element e in bits 16 (e % 2) of word e / 2).
__device__ __forceinline__ void split8(const float (&x)[8], u32x4& hi, u32x4& lo) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const floatx2 v = {x[2 * w], x[2 * w + 1]};
    const unsigned h = bf16_pair(v);
    const floatx2 hv = {__uint_as_float(h << 16), __uint_as_float(h & 0xffff0000u)};
    hi[w] = h;
    lo[w] = bf16_pair(v - hv);
  }
}

__device__ __forceinline__ bf16x8 as_bf16(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ floatx4 mfma(u32x4 a, u32x4 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16(a), as_bf16(b), c, 0, 0, 0);
}

// X rows of one wave as split srcB operands: xh[t], xl[t] = X[row0 + l16][32t + 8q .. + 7].
template <int RP>
__device__ __forceinline__ void load_x(u32x4 (&xh)[RP / 32], u32x4 (&xl)[RP / 32],
                                       const float* __restrict__ X, int64_t rows, int64_t row0,
                                       int q, int l16) {
  const int64_t row = row0 + l16;
#pragma unroll
  for (int t = 0; t < RP / 32; ++t) {
    float x[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (row < rows) {
      const float4 a = *reinterpret_cast<const float4*>(X + row * RP + 32 * t + 8 * q);
      const float4 b = *reinterpret_cast<const float4*>(X + row * RP + 32 * t + 8 * q + 4);
      x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
      x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
    }
    split8(x, xh[t], xl[t]);
  }
}

template <int RP>
struct Cfg32;

// Row-major tile of the 32-row form: rows unpadded, 16-byte chunk c of row j stored at
// c ^ swz32(j), which spreads 16 consecutive rows over 16 distinct bank groups for the first
// product's reads while letting one direct load cover 64 consecutive chunks (several rows).
template <int RP>
__device__ __forceinline__ int swz32(int row) {
  constexpr int C = RP / 4;  // chunks per row
  return C >= 16 ? (row & 15) : (C == 8 ? ((row >> 1) & 7) : ((row >> 2) & 3));
}

template <int RP>
__device__ __forceinline__ void stage32(float* dst, const float* __restrict__ rowm,
                                        const float* __restrict__ trans, int64_t j0, int64_t jb1,
                                        int wave, int lane) {
  using C = Cfg32<RP>;
  constexpr int CPR = RP / 4;
  constexpr int NI = C::NT * CPR / 64;  // direct loads of 64 chunks for the row-major tile
#pragma unroll
  for (int u = 0; u < NI / C::WAVES; ++u) {
    const int i = wave + C::WAVES * u;
    const int q = 64 * i + lane;           // chunk of the tile this lane fills
    const int r = q / CPR, ph = q - r * CPR;
    const int c = ph ^ swz32<RP>(r);       // logical chunk stored there
    const int64_t j = j0 + r;
    if (j < jb1)
      __builtin_amdgcn_global_load_lds((glb_void*)(rowm + j * RP + 4 * c),
                                       (lds_void*)(dst + 256 * i), 16, 0, 0);
    else
      *reinterpret_cast<float4*>(dst + 4 * q) = float4{0.f, 0.f, 0.f, 0.f};
  }
  const int64_t p0 = j0 / 32;
  const int64_t left = (jb1 - j0 + 31) / 32;
  const int np = left < C::NT / 32 ? (int)left : C::NT / 32;
  const int ninst = np * (C::TB / 256);
  float* tdst = dst + C::NT * C::LS;
  const float* tsrc = trans + p0 * C::TB;
  for (int i = wave; i < ninst; i += C::WAVES)
    __builtin_amdgcn_global_load_lds((glb_void*)(tsrc + 256 * i + 4 * lane),
                                     (lds_void*)(tdst + 256 * i), 16, 0, 0);
}

// 16 x 16 form: the rectified 16 x 32 tile (l0: panel rows 4q + v, l1: 16 + 4q + v) as the
// second product's split srcA operands, in the k order above; whether any of it is positive
// (wave-uniform).
__device__ __forceinline__ bool zsplit(floatx4 l0, floatx4 l1, u32x4& zh, u32x4& zl) {
  const float z[8] = {l0[0] > 0.f ? l0[0] : 0.f, l0[1] > 0.f ? l0[1] : 0.f,
                      l0[2] > 0.f ? l0[2] : 0.f, l0[3] > 0.f ? l0[3] : 0.f,
                      l1[0] > 0.f ? l1[0] : 0.f, l1[1] > 0.f ? l1[1] : 0.f,
                      l1[2] > 0.f ? l1[2] : 0.f, l1[3] > 0.f ? l1[3] : 0.f};
  split8(z, zh, zl);
  const bool pos = z[0] + z[1] + z[2] + z[3] + z[4] + z[5] + z[6] + z[7] > 0.f;
  return __ballot(pos) != 0;
}

// Panel rows of split s: [start(s), start(s + 1)), starts rounded down to whole pairs.
__host__ __device__ __forceinline__ int64_t pair_start(int s, int nsplit, int64_t blk) {
  return s >= nsplit ? blk : ((int64_t)s * blk / nsplit) / 32 * 32;
}

// ---------------------------------------------------------------------------------------------
// Ranks 32 to 128: 32 rows of X per wave on v_mfma_f32_32x32x16_bf16 (srcA lane l:
// A[l%32][8(l/32) + e], srcB lane l: B[8(l/32) + e][l%32], accumulator register v of lane l:
// D[8(v/4) + 4(l/32) + v%4][l%32]), which streams about 1.6 times the flops of the 16 x 16 x 32
// form.  Per 32-row panel block: the first product gives lane l the L^T values of X row l%32
// and panel rows j = 8(v/4) + 4(l/32) + v%4; rectified and split they are the srcA operands of
// two K = 16 MFMAs of the second product (a = 0, 1), k-slot (h, e) <-> panel row
// jrow32(a, h, e) = 16a + 8(e/4) + 4h + e%4.  The transposed panel copy holds, per block,
// [a][h][hi, lo][column] groups of those eight rows.

template <int RP>
struct Cfg32 {
  static constexpr int WAVES = 8;                     // two per SIMD
  static constexpr int ROWS = 32 * WAVES;             // rows of X per workgroup
  static constexpr int NT = RP >= 128 ? 64 : (RP >= 64 ? 128 : 256);
  static constexpr int LS = RP;                       // row-major rows unpadded, chunks swizzled
  static constexpr int RPC = RP < 32 ? 32 : RP;       // columns of the second product (r = 16
                                                      // pads to one 32-column block)
  static constexpr int TB = 32 * RPC;
  static constexpr int TILE = NT * LS + (NT / 32) * TB;
  static constexpr int CB = RPC / 32;                 // 32-column blocks of Y
  static_assert(RP % 16 == 0 && RP <= 128 && NT % WAVES == 0, "shape");
};

typedef __attribute__((ext_vector_type(16))) float floatx16;

__device__ __forceinline__ floatx16 mfma32(u32x4 a, u32x4 b, floatx16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16(a), as_bf16(b), c, 0, 0, 0);
}

__device__ __forceinline__ int jrow32(int a, int h, int e) {
  return 16 * a + 8 * (e >> 2) + 4 * h + (e & 3);
}

// Row-major and transposed split copies for the 32-row form (row-major: row j as RP/8 groups of
// 8 hi then 8 lo bf16; the transposed blocks are Cfg32<RP>::RPC columns wide, zero past RP).
template <int RP>
__global__ __launch_bounds__(256) void bx32_split_kernel(const float* __restrict__ P, int64_t blk,
                                                         int64_t npair, u32x4* __restrict__ rowm,
                                                         u32x4* __restrict__ trans) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t na = blk * (RP / 8);
  if (gid < na) {
    const int64_t row = gid / (RP / 8);
    const int g = (int)(gid - row * (RP / 8));
    const float4 a = *reinterpret_cast<const float4*>(P + row * RP + 8 * g);
    const float4 b = *reinterpret_cast<const float4*>(P + row * RP + 8 * g + 4);
    const float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    u32x4 hi, lo;
    split8(x, hi, lo);
    rowm[row * (RP / 4) + 2 * g] = hi;
    rowm[row * (RP / 4) + 2 * g + 1] = lo;
    return;
  }
  constexpr int RPC = Cfg32<RP>::RPC;
  const int64_t t = gid - na;
  if (t >= npair * 4 * RPC) return;
  const int64_t p = t / (4 * RPC);
  const int rem = (int)(t - p * 4 * RPC);
  const int ah = rem / RPC, c = rem - ah * RPC;  // ah = 2a + h
  float x[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int64_t j = 32 * p + jrow32(ah >> 1, ah & 1, e);
    x[e] = j < blk && c < RP ? P[j * RP + c] : 0.f;
  }
  u32x4 hi, lo;
  split8(x, hi, lo);
  u32x4* blkp = trans + p * (8 * RPC);
  blkp[(2 * ah) * RPC + c] = hi;
  blkp[(2 * ah + 1) * RPC + c] = lo;
}

// X rows of one wave as split srcB operands: xh[t], xl[t] = X[row0 + l%32][16t + 8h .. + 7].
template <int RP>
__device__ __forceinline__ void load_x32(u32x4 (&xh)[RP / 16], u32x4 (&xl)[RP / 16],
                                         const float* __restrict__ X, int64_t rows, int64_t row0,
                                         int h, int l32) {
  const int64_t row = row0 + l32;
#pragma unroll
  for (int t = 0; t < RP / 16; ++t) {
    float x[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (row < rows) {
      const float4 a = *reinterpret_cast<const float4*>(X + row * RP + 16 * t + 8 * h);
      const float4 b = *reinterpret_cast<const float4*>(X + row * RP + 16 * t + 8 * h + 4);
      x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
      x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
    }
    split8(x, xh[t], xl[t]);
  }
}

// First product of panel block jp: L^T (32 panel rows x 32 X rows) in two accumulator chains.
template <int RP>
__device__ __forceinline__ floatx16 gemm1_blk32(const float* tile, int jp,
                                                const u32x4 (&xh)[RP / 16],
                                                const u32x4 (&xl)[RP / 16], int h, int l32) {
  using C = Cfg32<RP>;
  constexpr int KC = RP / 16;
  constexpr int LA = RP >= 128 ? 1 : (KC < 2 ? KC : 2);  // one chunk ahead where registers are short
  const int row = 32 * jp + l32;
  const u32x4* pr = reinterpret_cast<const u32x4*>(tile + row * C::LS);
  const int sw = swz32<RP>(row);
  floatx16 a0, a1;
#pragma unroll
  for (int v = 0; v < 16; ++v) a0[v] = a1[v] = 0.f;
  u32x4 ph[KC], pl[KC];
#pragma unroll
  for (int t = 0; t < LA; ++t) {
    ph[t] = pr[(2 * (2 * t + h)) ^ sw];
    pl[t] = pr[(2 * (2 * t + h) + 1) ^ sw];
  }
#pragma unroll
  for (int t = 0; t < KC; ++t) {
    if (t + LA < KC) {
      ph[t + LA] = pr[(2 * (2 * (t + LA) + h)) ^ sw];
      pl[t + LA] = pr[(2 * (2 * (t + LA) + h) + 1) ^ sw];
    }
    a0 = mfma32(ph[t], xh[t], a0);
    a1 = mfma32(ph[t], xl[t], a1);
    a0 = mfma32(pl[t], xh[t], a0);
    __builtin_amdgcn_sched_barrier(0);
  }
  return a0 + a1;
}

// Ranks up to 32 (at most two k chunks): a block's panel operands as registers, read a block
// ahead of its MFMAs, so that the LDS latency hides behind the previous block's work.
template <int RP>
struct Ops32 {
  u32x4 h[RP / 16], l[RP / 16];
};

template <int RP>
__device__ __forceinline__ void load_blk32(Ops32<RP>& o, const float* tile, int jp, int h,
                                           int l32) {
  const int row = 32 * jp + l32;
  const u32x4* pr = reinterpret_cast<const u32x4*>(tile + row * Cfg32<RP>::LS);
  const int sw = swz32<RP>(row);
#pragma unroll
  for (int t = 0; t < RP / 16; ++t) {
    o.h[t] = pr[(2 * (2 * t + h)) ^ sw];
    o.l[t] = pr[(2 * (2 * t + h) + 1) ^ sw];
  }
}

template <int RP>
__device__ __forceinline__ floatx16 mma_blk32(const Ops32<RP>& o, const u32x4 (&xh)[RP / 16],
                                              const u32x4 (&xl)[RP / 16]) {
  // one accumulator chain: at r_p <= 32 it is at most six MFMAs long, and adding two chains
  // would cost 16 vector adds per block in a kernel that is bound by its vector work
  floatx16 a0;
#pragma unroll
  for (int v = 0; v < 16; ++v) a0[v] = 0.f;
#pragma unroll
  for (int t = 0; t < RP / 16; ++t) {
    a0 = mfma32(o.h[t], xh[t], a0);
    a0 = mfma32(o.h[t], xl[t], a0);
    a0 = mfma32(o.l[t], xh[t], a0);
  }
  return a0;
}

// Rectified block as the second product's split srcA operands (a = 0: registers 0..7,
// a = 1: registers 8..15); whether any of it is positive (wave-uniform).
__device__ __forceinline__ bool zsplit32(floatx16 l, u32x4 (&zh)[2], u32x4 (&zl)[2]) {
  float z[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) z[v] = l[v] > 0.f ? l[v] : 0.f;
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    float x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = z[8 * a + e];
    split8(x, zh[a], zl[a]);
  }
  // live when any hi part is nonzero (a value whose hi part rounds to zero has a zero lo part
  // too, so it adds nothing to the second product)
  const unsigned any = (zh[0][0] | zh[0][1]) | (zh[0][2] | zh[0][3]) | (zh[1][0] | zh[1][1]) |
                       (zh[1][2] | zh[1][3]);
  return __ballot(any != 0u) != 0;
}

// Second product of block jp into the 32 x 32 tiles of Y; with NEXT the next block's rectify
// and split (from ln) is placed after the first column block, so that its vector work issues
// while the MFMAs run.
template <int RP, bool NEXT>
__device__ __forceinline__ bool gemm2_blk32(floatx16 (&y)[Cfg32<RP>::CB], floatx16& y2,
                                            const float* trans, int jp, const u32x4 (&zh)[2],
                                            const u32x4 (&zl)[2], floatx16 ln, u32x4 (&nzh)[2],
                                            u32x4 (&nzl)[2], int h, int l32) {
  using C = Cfg32<RP>;
  constexpr int CB = C::CB;
  const u32x4* base = reinterpret_cast<const u32x4*>(trans + jp * C::TB) + l32;
  bool live = false;
  if constexpr (CB == 1) {
    // one column block: the a = 1 half accumulates into y2 so that the two chains interleave
    u32x4 bh[2], bl[2];
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      bh[a] = base[(2 * (2 * a + h)) * C::RPC];
      bl[a] = base[(2 * (2 * a + h) + 1) * C::RPC];
    }
    y[0] = mfma32(zh[0], bh[0], y[0]);
    y2 = mfma32(zh[1], bh[1], y2);
    y[0] = mfma32(zh[0], bl[0], y[0]);
    y2 = mfma32(zh[1], bl[1], y2);
    y[0] = mfma32(zl[0], bh[0], y[0]);
    y2 = mfma32(zl[1], bh[1], y2);
    if (NEXT) live = zsplit32(ln, nzh, nzl);
    return live;
  }
#pragma unroll
  for (int cb = 0; cb < CB; ++cb) {
    u32x4 bh[2], bl[2];
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      bh[a] = base[(2 * (2 * a + h)) * C::RPC + 32 * cb];
      bl[a] = base[(2 * (2 * a + h) + 1) * C::RPC + 32 * cb];
    }
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      y[cb] = mfma32(zh[a], bh[a], y[cb]);
      y[cb] = mfma32(zh[a], bl[a], y[cb]);
      y[cb] = mfma32(zl[a], bh[a], y[cb]);
    }
    if (NEXT && cb == 0) live = zsplit32(ln, nzh, nzl);
  }
  return live;
}

template <int RP>
__device__ __forceinline__ unsigned consume32(const float* tile, int np,
                                              const u32x4 (&xh)[RP / 16],
                                              const u32x4 (&xl)[RP / 16],
                                              floatx16 (&y)[Cfg32<RP>::CB], floatx16& y2, int h,
                                              int l32) {
  using C = Cfg32<RP>;
  const float* trans = tile + C::NT * C::LS;
  unsigned ran = 0;
  u32x4 zh[2], zl[2];
  if constexpr (RP >= 128) {
    // two waves per SIMD leave no registers for the pipelined form: one block at a time
    floatx16 zero;
#pragma unroll
    for (int v = 0; v < 16; ++v) zero[v] = 0.f;
    for (int jp = 0; jp < np; ++jp) {
      if (zsplit32(gemm1_blk32<RP>(tile, jp, xh, xl, h, l32), zh, zl)) {
        u32x4 dh[2], dl[2];
        gemm2_blk32<RP, false>(y, y2, trans, jp, zh, zl, zero, dh, dl, h, l32);
        ++ran;
      }
    }
    return ran;
  }
  if constexpr (RP <= 32) {
    // operands a block ahead in ping-pong registers: the reads of block jp + 2 are in flight
    // during the second product of block jp
    Ops32<RP> o0, o1;  // block jp's operands alternate between o0 (even) and o1 (odd)
    load_blk32<RP>(o0, tile, 0, h, l32);
    if (np > 1) load_blk32<RP>(o1, tile, 1, h, l32);
    bool live = zsplit32(mma_blk32<RP>(o0, xh, xl), zh, zl);
    // one block: the first product of jp + 1 (operands in nxt), the reads of jp + 2 (into
    // reload, whose block jp is done), the second product of jp with the split of jp + 1
    auto block = [&](int jp, const Ops32<RP>& nxt, Ops32<RP>& reload) {
      floatx16 ln;
#pragma unroll
      for (int v = 0; v < 16; ++v) ln[v] = 0.f;
      if (jp + 1 < np) ln = mma_blk32<RP>(nxt, xh, xl);
      if (jp + 2 < np) load_blk32<RP>(reload, tile, jp + 2, h, l32);
      u32x4 nzh[2], nzl[2];
      bool nlive;
      if (live) {
        nlive = gemm2_blk32<RP, true>(y, y2, trans, jp, zh, zl, ln, nzh, nzl, h, l32);
        ++ran;
      } else {
        nlive = zsplit32(ln, nzh, nzl);
      }
#pragma unroll
      for (int a = 0; a < 2; ++a) {
        zh[a] = nzh[a];
        zl[a] = nzl[a];
      }
      live = nlive;
    };
    for (int jp = 0; jp < np; jp += 2) {
      block(jp, o1, o0);
      if (jp + 1 < np) block(jp + 1, o0, o1);
    }
    return ran;
  }
  bool live = zsplit32(gemm1_blk32<RP>(tile, 0, xh, xl, h, l32), zh, zl);
  for (int jp = 0; jp < np; ++jp) {
    floatx16 ln;
#pragma unroll
    for (int v = 0; v < 16; ++v) ln[v] = 0.f;
    if (jp + 1 < np) ln = gemm1_blk32<RP>(tile, jp + 1, xh, xl, h, l32);
    u32x4 nzh[2], nzl[2];
    bool nlive;
    if (live) {
      nlive = gemm2_blk32<RP, true>(y, y2, trans, jp, zh, zl, ln, nzh, nzl, h, l32);
      ++ran;
    } else {
      nlive = zsplit32(ln, nzh, nzl);
    }
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      zh[a] = nzh[a];
      zl[a] = nzl[a];
    }
    live = nlive;
  }
  return ran;
}

template <int RP>
__device__ __forceinline__ unsigned step32(const float* __restrict__ cur, float* __restrict__ nxt,
                                           const float* __restrict__ rowm,
                                           const float* __restrict__ trans, int64_t j0,
                                           int64_t jb1, const u32x4 (&xh)[RP / 16],
                                           const u32x4 (&xl)[RP / 16], floatx16 (&y)[Cfg32<RP>::CB],
                                           floatx16& y2, int wave, int lane, int h, int l32) {
  constexpr int NT = Cfg32<RP>::NT;
  if (nxt) stage32<RP>(nxt, rowm, trans, j0 + NT, jb1, wave, lane);
  const int64_t left = (jb1 - j0 + 31) / 32;
  return consume32<RP>(cur, left < NT / 32 ? (int)left : NT / 32, xh, xl, y, y2, h, l32);
}

template <int RP>
__global__ __launch_bounds__(64 * Cfg32<RP>::WAVES) void bx32_kernel(
    const float* __restrict__ X, int64_t rows, const float* __restrict__ rowm,
    const float* __restrict__ trans, int64_t blk, float* __restrict__ Ypart, int64_t y_stride,
    int nsplit, int64_t row_tiles, float sgn, unsigned long long* __restrict__ live_slices) {
  using C = Cfg32<RP>;
  constexpr int CB = C::CB;
  __shared__ __attribute__((aligned(16))) float smem[2 * C::TILE];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5, l32 = lane & 31;

  const int64_t logical = xcd_logical(blockIdx.x, (int64_t)gridDim.x);
  const int split = (int)(logical / row_tiles);
  const int64_t rt = logical - (int64_t)split * row_tiles;
  const int64_t jb0 = pair_start(split, nsplit, blk);
  const int64_t jb1 = pair_start(split + 1, nsplit, blk);
  const int64_t row0 = rt * C::ROWS + (int64_t)wave * 32;

  u32x4 xh[RP / 16], xl[RP / 16];
  load_x32<RP>(xh, xl, X, rows, row0, h, l32);
  floatx16 y[CB], y2;  // y2: second accumulator of the one-column-block case
#pragma unroll
  for (int v = 0; v < 16; ++v) y2[v] = 0.f;
#pragma unroll
  for (int cb = 0; cb < CB; ++cb)
#pragma unroll
    for (int v = 0; v < 16; ++v) y[cb][v] = 0.f;

  if (jb0 < jb1) stage32<RP>(smem, rowm, trans, jb0, jb1, wave, lane);
  int cur = 0;
  unsigned ran = 0;
  for (int64_t j0 = jb0; j0 < jb1; j0 += C::NT, cur ^= 1) {
    __builtin_amdgcn_s_waitcnt(0);  // this wave's loads of the tile have landed
    __syncthreads();                // every wave's have; the other buffer is free again
    ran += step32<RP>(smem + cur * C::TILE, j0 + C::NT < jb1 ? smem + (cur ^ 1) * C::TILE : nullptr,
                      rowm, trans, j0, jb1, xh, xl, y, y2, wave, lane, h, l32);
  }
  if constexpr (CB == 1) y[0] += y2;

  float* Y = Ypart + (int64_t)split * y_stride;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int64_t row = row0 + 8 * (v / 4) + 4 * h + (v % 4);
    if (row < rows) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
        if (RP % 32 == 0 || 32 * cb + l32 < RP) Y[row * RP + 32 * cb + l32] = sgn * y[cb][v];
    }
  }
  // a live 32 x 32 tile counts as its sixteen 16 x 4 slices of max(0, L)
  if (live_slices && lane == 0 && ran) atomicAdd(live_slices, 16ull * ran);
}

}  // namespace bx

// Launchers: the panel split, then the contraction kernel over row_tiles x nsplit workgroups.
template <int RP>
static hipError_t bx32_launch_t(const float* X, int64_t rows, const float* P, int64_t blk,
                                float* work, float* Ypart, int64_t y_stride, int nsplit,
                                float sgn, unsigned long long* live, hipStream_t st) {
  using C = bx::Cfg32<RP>;
  const int64_t npair = (blk + 31) / 32;
  float* rowm = work;
  float* trans = work + blk * RP;
  const int64_t threads = blk * (RP / 8) + npair * 4 * C::RPC;
  hipLaunchKernelGGL(bx::bx32_split_kernel<RP>, dim3((unsigned)((threads + 255) / 256)),
                     dim3(256), 0, st, P, blk, npair, reinterpret_cast<bx::u32x4*>(rowm),
                     reinterpret_cast<bx::u32x4*>(trans));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t row_tiles = (rows + C::ROWS - 1) / C::ROWS;
  const int64_t total = row_tiles * nsplit;
  if (total <= 0) return hipSuccess;
  if (total > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(bx::bx32_kernel<RP>, dim3((unsigned)total), dim3(64 * C::WAVES), 0, st, X,
                     rows, rowm, trans, blk, Ypart, y_stride, nsplit, row_tiles, sgn, live);
  return hipGetLastError();
}

}  // namespace nmd
