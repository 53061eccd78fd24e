// Split-bf16 variant of the fused dense contraction at r_p = 256 (an option beside the fp32
// kernel): the first product L = X P^T runs on bf16 MFMA with every operand split in two,
// x = x_hi + x_lo (x_hi = bf16(x), x_lo = bf16(x - x_hi), 16 significant bits in all), and
// L = X_hi P_hi^T + X_hi P_lo^T + X_lo P_hi^T accumulated in fp32 (the dropped X_lo P_lo^T and
// the split remainders are of relative size 2^-16).  This is the gfx950 counterpart of the
// paper's TF32 kernels (Sec. 4.2): gfx950 has no TF32 matrix instructions, and bf16 MFMA runs at
// 16 times the fp32 rate, so the three products cost about a fifth of the fp32 first product.
// Everything after L is the fp32 kernel's: rectify in registers, skip zero 16 x 4 slices, pack
// thin slices into gathered slices, run the rest whole; the second product's srcB values are
// read back from the split panel as p_hi + p_lo.
//
// Operands (v_mfma_f32_16x16x32_bf16, one 16 x 16 L^T tile per 32-wide k chunk t): srcA lane
// (q, l16) holds panel row l16 of the j-block, k = 32t + 8q .. 32t + 8q + 7; srcB holds X row
// l16, the same k.  The accumulator then has lane (q, l16), register v = L[i = l16][j = 4q + v],
// the layout of the fp32 kernel.  The panel is split once per step by split_panel_kernel into
// rows of 32 groups of (8 hi, 8 lo) bf16 (1 KB per row), so one ds_read_b128 reads one operand.

#pragma once

#include "dense_kernel.h"

namespace nmd {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) unsigned uintx4;

// bf16 of x, rounded to nearest even (finite x).
__device__ __forceinline__ unsigned bf16_bits(float x) {
  const unsigned u = __float_as_uint(x);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ float bf16_value(unsigned h) { return __uint_as_float(h << 16); }

// Eight consecutive values split into packed hi and lo halves (element e in bits 16(e%2) of
// word e/2).
__device__ __forceinline__ void split8(const float (&x)[8], uintx4& hi, uintx4& lo) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const unsigned h0 = bf16_bits(x[2 * w]), h1 = bf16_bits(x[2 * w + 1]);
    const unsigned l0 = bf16_bits(x[2 * w] - bf16_value(h0));
    const unsigned l1 = bf16_bits(x[2 * w + 1] - bf16_value(h1));
    hi[w] = h0 | (h1 << 16);
    lo[w] = l0 | (l1 << 16);
  }
}

// One split panel row (256 values) per 32 threads: thread g writes group g = 8 values as
// (8 hi, 8 lo), 32 bytes.  rows x 1 KB out.
__global__ __launch_bounds__(256) void split_panel_kernel(const float* __restrict__ P,
                                                          int64_t rows, uintx4* __restrict__ out) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= rows * 32) return;
  const int64_t row = gid >> 5;
  const int g = (int)(gid & 31);
  const float4 a = *reinterpret_cast<const float4*>(P + row * 256 + 8 * g);
  const float4 b = *reinterpret_cast<const float4*>(P + row * 256 + 8 * g + 4);
  const float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  uintx4 hi, lo;
  split8(x, hi, lo);
  out[row * 64 + 2 * g] = hi;
  out[row * 64 + 2 * g + 1] = lo;
}

// X rows of one wave as split srcB operands: xh[t], xl[t] = X[row0 + l16][32t + 8q .. + 7].
__device__ __forceinline__ void load_x_split(uintx4 (&xh)[8], uintx4 (&xl)[8],
                                             const float* __restrict__ X, int64_t rows,
                                             int64_t row0, int q, int l16) {
  const int64_t row = row0 + l16;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    float x[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (row < rows) {
      const float4 a = *reinterpret_cast<const float4*>(X + row * 256 + 32 * t + 8 * q);
      const float4 b = *reinterpret_cast<const float4*>(X + row * 256 + 32 * t + 8 * q + 4);
      x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
      x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
    }
    split8(x, xh[t], xl[t]);
  }
}

__device__ __forceinline__ bf16x8 as_bf16x8(uintx4 v) { return __builtin_bit_cast(bf16x8, v); }

// L^T tile of j-block jb from the split panel tile (LDS rows of 1 KB at a stride of 260 floats).
// Three accumulator chains (hi hi, hi lo, lo hi); the reads run two chunks ahead.
__device__ __forceinline__ void l_tile_split(floatx4& lt, const uintx4 (&xh)[8],
                                             const uintx4 (&xl)[8], const float* tile, int jb,
                                             int q, int l16) {
  constexpr int LS = 260;
  const uintx4* prow = reinterpret_cast<const uintx4*>(tile + (jb * 16 + l16) * LS);
  floatx4 acc[3] = {floatx4{0.f, 0.f, 0.f, 0.f}, floatx4{0.f, 0.f, 0.f, 0.f},
                    floatx4{0.f, 0.f, 0.f, 0.f}};
  uintx4 ph[8], pl[8];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    ph[t] = prow[2 * (4 * t + q)];
    pl[t] = prow[2 * (4 * t + q) + 1];
  }
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    if (t + 2 < 8) {
      ph[t + 2] = prow[2 * (4 * (t + 2) + q)];
      pl[t + 2] = prow[2 * (4 * (t + 2) + q) + 1];
    }
    acc[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ph[t]), as_bf16x8(xh[t]), acc[0], 0, 0, 0);
    acc[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ph[t]), as_bf16x8(xl[t]), acc[1], 0, 0, 0);
    acc[2] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(pl[t]), as_bf16x8(xh[t]), acc[2], 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
  lt = acc[0] + (acc[1] + acc[2]);
}

// fp32 value hi + lo of column c of a split panel row (u16 units: group c/8 at 16 (c/8), hi at
// + c%8, lo at + 8 + c%8).
__device__ __forceinline__ float split_value(const unsigned short* row, int c) {
  const int base = 16 * (c >> 3) + (c & 7);
  return bf16_value(row[base]) + bf16_value(row[base + 8]);
}

// srcB of slice v of j-block jb for the second product: P[jb*16 + 4q + v][16 cb + l16].
__device__ __forceinline__ void zb_read_split(float (&bb)[16], const float* tile, int jb, int v,
                                              int q, int l16) {
  const unsigned short* row =
      reinterpret_cast<const unsigned short*>(tile + (jb * 16 + 4 * q + v) * 260);
#pragma unroll
  for (int cb = 0; cb < 16; ++cb) bb[cb] = split_value(row, 16 * cb + l16);
}

// One gathered slice from the `cnt` (1..4) list entries at head .. head + cnt - 1, with the
// panel rows read from a split tile.
__device__ __forceinline__ void elist_slice_split(floatx4 (&y)[16], const uint2* el, unsigned head,
                                                  int cnt, const float* tile, int q, int l16) {
  const uint2 e = el[(head + q) % ELIST];
  const bool valid = q < cnt;
  const int row = valid ? (int)(e.x >> 4) : 0;
  const float a = valid && l16 == (int)(e.x & 15u) ? __uint_as_float(e.y) : 0.f;
  const unsigned short* prow = reinterpret_cast<const unsigned short*>(tile + row * 260);
  float bb[16];
#pragma unroll
  for (int cb = 0; cb < 16; ++cb) bb[cb] = split_value(prow, 16 * cb + l16);
#pragma unroll
  for (int cb = 0; cb < 16; ++cb)
    y[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bb[cb], y[cb], 0, 0, 0);
}

// Both products over the split panel rows j0 .. min(j0 + 64, jb1) - 1 (the fp32 kernel's
// r_p = 256 path with the split first product).
__device__ __forceinline__ unsigned consume_tile_split(const float* tile, int64_t j0, int64_t jb1,
                                                       const uintx4 (&xh)[8],
                                                       const uintx4 (&xl)[8], floatx4 (&y)[16],
                                                       int q, int l16, unsigned& entries,
                                                       uint2* el) {
  constexpr int SPARSE = DenseLaunch<256>::SPARSE;
  const int left = (int)((jb1 - j0 + 15) / 16);
  const int njb = left < 4 ? left : 4;
  unsigned done = 0;
  unsigned head = 0, tail = 0;
  for (int jb = 0; jb < njb; ++jb) {
    floatx4 lt;
    l_tile_split(lt, xh, xl, tile, jb, q, l16);
#pragma unroll
    for (int v = 0; v < 4; ++v) lt[v] = lt[v] > 0.f ? lt[v] : 0.f;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const unsigned long long bits = __ballot(lt[v] > 0.f);
      if (!bits) continue;
      const int cnt = __popcll(bits);
      if (cnt <= SPARSE) {
        elist_push(el, tail, bits, lt[v], jb, v, q, l16);
        tail += cnt;
        entries += cnt;
      } else {
        float bb[16];
        zb_read_split(bb, tile, jb, v, q, l16);
#pragma unroll
        for (int cb = 0; cb < 16; ++cb)
          y[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(lt[v], bb[cb], y[cb], 0, 0, 0);
        ++done;
      }
    }
    for (; tail - head >= 4; head += 4) elist_slice_split(y, el, head, 4, tile, q, l16);
  }
  if (tail != head) elist_slice_split(y, el, head, (int)(tail - head), tile, q, l16);
  return done;
}

__device__ __forceinline__ unsigned split_step(const float* __restrict__ cur, float* __restrict__ nxt,
                                               const float* __restrict__ P, int64_t j0,
                                               int64_t jb1, const uintx4 (&xh)[8],
                                               const uintx4 (&xl)[8], floatx4 (&y)[16], int wave,
                                               int lane, int q, int l16, unsigned& entries,
                                               uint2* el) {
  if (nxt) issue_tile<256>(nxt, P, j0 + DenseLaunch<256>::NT, jb1, wave, lane);
  return consume_tile_split(cur, j0, jb1, xh, xl, y, q, l16, entries, el);
}

// Y_s = sgn * max(0, X P^T) P at r_p = 256 with the split first product; Psplit holds the
// panel rows split by split_panel_kernel (1 KB per row), otherwise as dense_kernel<256>.
__global__ __launch_bounds__(64 * DenseLaunch<256>::WAVES) void dense_split_kernel(
    const float* __restrict__ X, int64_t rows, const float* __restrict__ Psplit, int64_t blk,
    float* __restrict__ Ypart, int64_t y_stride, int nsplit, int64_t row_tiles, float sgn,
    unsigned long long* __restrict__ gemm2_blocks) {
  constexpr int WAVES = DenseLaunch<256>::WAVES;
  constexpr int NT = DenseLaunch<256>::NT;
  constexpr int LS = 260;
  __shared__ __attribute__((aligned(16))) float smem[2 * NT * LS];
  __shared__ uint2 elists[WAVES * ELIST];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q = lane >> 4, l16 = lane & 15;
  uint2* el = &elists[wave * ELIST];

  const int64_t logical = xcd_logical(blockIdx.x, (int64_t)gridDim.x);
  const int split = (int)(logical / row_tiles);
  const int64_t rt = logical - (int64_t)split * row_tiles;
  const int64_t jb0 = (int64_t)split * blk / nsplit;
  const int64_t jb1 = (int64_t)(split + 1) * blk / nsplit;
  const int64_t row0 = rt * dense_rows<256>() + (int64_t)wave * 16;

  uintx4 xh[8], xl[8];
  load_x_split(xh, xl, X, rows, row0, q, l16);

  floatx4 y[16];
#pragma unroll
  for (int cb = 0; cb < 16; ++cb) y[cb] = floatx4{0.f, 0.f, 0.f, 0.f};

  unsigned done = 0, entries = 0;
  if (jb0 < jb1) issue_tile<256>(smem, Psplit, jb0, jb1, wave, lane);
  int cur = 0;
  for (int64_t j0 = jb0; j0 < jb1; j0 += NT, cur ^= 1) {
    __builtin_amdgcn_s_waitcnt(0);  // this wave's loads of the tile have landed
    __syncthreads();                // every wave's have; the other buffer is free again
    done += split_step(smem + cur * (NT * LS), j0 + NT < jb1 ? smem + (cur ^ 1) * (NT * LS) : nullptr,
                       Psplit, j0, jb1, xh, xl, y, wave, lane, q, l16, entries, el);
  }

  float* Y = Ypart + (int64_t)split * y_stride;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int64_t row = row0 + 4 * q + v;
    if (row < rows) {
#pragma unroll
      for (int cb = 0; cb < 16; ++cb) Y[row * 256 + 16 * cb + l16] = sgn * y[cb][v];
    }
  }
  if (gemm2_blocks && lane == 0) {
    atomicAdd(gemm2_blocks, (unsigned long long)done);
    if (entries) atomicAdd(gemm2_blocks + 1, (unsigned long long)entries);
  }
}

}  // namespace nmd
