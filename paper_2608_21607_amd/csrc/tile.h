// Device building blocks shared by the fused contraction and the objective kernels:
// per-rank tiling constants, the XCD-aware workgroup order, the resident X fragments, the LDS
// panel tile and the transposed L tile on v_mfma_f32_16x16x4f32.
#pragma once

#include "nmd_internal.h"

namespace nmd {

typedef float floatx4 __attribute__((ext_vector_type(4)));

template <int RP>
struct DenseCfg;
// MI: 16-row blocks of X per wave (4 waves per workgroup).  NT: panel rows per LDS tile.
// NT: panel rows per register-staged LDS tile (objective kernel).  NTD: panel rows per
// directly loaded, double-buffered LDS tile of the contraction (a multiple of 16; both buffers
// together within the 160 KB of LDS).
template <> struct DenseCfg<16>  { static constexpr int MI = 4, NT = 512, NTD = 512; };
template <> struct DenseCfg<32>  { static constexpr int MI = 4, NT = 256, NTD = 512; };
template <> struct DenseCfg<48>  { static constexpr int MI = 4, NT = 160, NTD = 320; };
template <> struct DenseCfg<64>  { static constexpr int MI = 4, NT = 128, NTD = 256; };
template <> struct DenseCfg<128> { static constexpr int MI = 4, NT = 64, NTD = 128; };
template <> struct DenseCfg<192> { static constexpr int MI = 2, NT = 32, NTD = 80; };
template <> struct DenseCfg<256> { static constexpr int MI = 2, NT = 32, NTD = 64; };
template <> struct DenseCfg<320> { static constexpr int MI = 1, NT = 16, NTD = 48; };
template <> struct DenseCfg<384> { static constexpr int MI = 1, NT = 16, NTD = 32; };
template <> struct DenseCfg<448> { static constexpr int MI = 1, NT = 16, NTD = 32; };
template <> struct DenseCfg<512> { static constexpr int MI = 1, NT = 16, NTD = 32; };

template <int RP>
constexpr int rows_per_wg() { return 64 * DenseCfg<RP>::MI; }

// Workgroups are dispatched round-robin over the 8 XCDs; this maps the hardware index to a
// logical one so that XCD x (= bid % 8) owns a contiguous range of logical indices.
__device__ __forceinline__ int64_t xcd_logical(int64_t bid, int64_t total) {
  const int64_t x = bid & 7, local = bid >> 3;
  const int64_t per = total >> 3, rem = total & 7;
  return x * per + (x < rem ? x : rem) + local;
}

// Resident X fragments: a[mi][4t + c] = X[row0 + 16 mi + l16][16t + 4q + c] (zero past rows).
template <int RP, int MI>
__device__ __forceinline__ void load_x_frags(float (&a)[MI][RP / 4], const float* __restrict__ X,
                                             int64_t rows, int64_t row0, int q, int l16) {
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
    const int64_t row = row0 + 16 * mi + l16;
#pragma unroll
    for (int t = 0; t < RP / 16; ++t) {
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (row < rows) v = *reinterpret_cast<const float4*>(X + row * RP + 16 * t + 4 * q);
      a[mi][4 * t + 0] = v.x;
      a[mi][4 * t + 1] = v.y;
      a[mi][4 * t + 2] = v.z;
      a[mi][4 * t + 3] = v.w;
    }
  }
}

// Panel tile staging: NT rows of P (row stride RP) into LDS with row stride RP + 4 by THREADS
// threads; rows at or past `jend` are zero.  fetch() issues the global loads into registers,
// stash() stores them.
template <int RP, int NT_, int THREADS = 256>
struct PanelTile {
  static constexpr int NT = NT_;
  static constexpr int LS = RP + 4;
  static constexpr int NV4 = NT * RP / 4;
  static constexpr int NLD = (NV4 + THREADS - 1) / THREADS;
  float4 pf[NLD];

  __device__ __forceinline__ void fetch(const float* __restrict__ P, int64_t j0, int64_t jend,
                                        int tid) {
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int f = tid + THREADS * u;
      const int rr = f / (RP / 4), c4 = f - rr * (RP / 4);
      const int64_t j = j0 + rr;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (f < NV4 && j < jend) v = *reinterpret_cast<const float4*>(P + j * RP + 4 * c4);
      pf[u] = v;
    }
  }
  __device__ __forceinline__ void stash(float* tile, int tid) const {
#pragma unroll
    for (int u = 0; u < NLD; ++u) {
      const int f = tid + THREADS * u;
      const int rr = f / (RP / 4), c4 = f - rr * (RP / 4);
      if (f < NV4) *reinterpret_cast<float4*>(&tile[rr * LS + 4 * c4]) = pf[u];
    }
  }
};

// Fragment groups of the panel read ahead of the first product's MFMAs.
template <int RP>
constexpr int l_lookahead() { return RP / 16 < 3 ? RP / 16 : 3; }

// The first l_lookahead<RP>() fragment groups of j-block jb, read before the block's MFMAs
// start (typically while the previous block's second product runs).
template <int RP>
__device__ __forceinline__ void l_prefetch(float4 (&pre)[l_lookahead<RP>()], const float* tile,
                                           int jb, int q, int l16) {
  const float* brow = &tile[(jb * 16 + l16) * (RP + 4) + 4 * q];
#pragma unroll
  for (int t = 0; t < l_lookahead<RP>(); ++t) pre[t] = *reinterpret_cast<const float4*>(brow + 16 * t);
}

// Accumulator chains of the first product (NA below).
template <int MI>
constexpr int l_chains() { return MI >= 2 ? 1 : 2; }

// Transposed L tile of one 16-row j-block: lt[mi] lane l, register v holds
// L[i = row0 + 16 mi + l16][j = jb*16 + 4q + v] (srcA = panel rows, srcB = X rows, both over
// the permuted k order 16t + 4q + c, one ds_read_b128 per four k-steps).  `pre` holds the first
// fragment groups (l_prefetch).  Each k-group issues, in this order and fenced from the next
// group: the read of group t + LA, its share of the srcB operands of the block's second product
// (the NR slices of `ring`, NR = 0, 2 or 4), then its MFMAs, which take the NA accumulators
// round-robin per k-step so that dependent MFMAs are at least two apart.
// l_tile_acc leaves the NA chains unsummed (acc[h][mi], lt[mi] = sum over h), so that a caller
// can hold them past the next block's MFMAs before it needs their sum.
template <int RP, int MI, int NR>
__device__ __forceinline__ void l_tile_acc(floatx4 (&acc)[l_chains<MI>()][MI],
                                           const float (&a)[MI][RP / 4],
                                           const float4 (&pre)[l_lookahead<RP>()],
                                           float (&ring)[NR > 0 ? NR : 1][RP / 16],
                                           const float* tile, int jb, int q, int l16) {
  constexpr int LS = RP + 4;
  constexpr int KG = RP / 16;
  constexpr int CB = RP / 16;
  constexpr int LA = l_lookahead<RP>();
  constexpr int NA = l_chains<MI>();
  constexpr int PER = NR * CB / KG;  // ring values read per k-group (NR * CB = NR * KG)
#pragma unroll
  for (int h = 0; h < NA; ++h)
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) acc[h][mi] = floatx4{0.f, 0.f, 0.f, 0.f};
  const float* brow = &tile[(jb * 16 + l16) * LS + 4 * q];
  const float* b2 = &tile[(jb * 16 + 4 * q) * LS + l16];
  float4 bf[KG];
#pragma unroll
  for (int t = 0; t < LA; ++t) bf[t] = pre[t];
#pragma unroll
  for (int t = 0; t < KG; ++t) {
    if (t + LA < KG)
      bf[t + LA] = *reinterpret_cast<const float4*>(brow + 16 * (t + LA));
    if constexpr (NR > 0) {
#pragma unroll
      for (int e = PER * t; e < PER * t + PER; ++e)
        ring[e / CB][e % CB] = b2[(e / CB) * LS + 16 * (e % CB)];
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int h = (4 * t + c) % NA;
      const float bk = c == 0 ? bf[t].x : c == 1 ? bf[t].y : c == 2 ? bf[t].z : bf[t].w;
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
        acc[h][mi] = __builtin_amdgcn_mfma_f32_16x16x4f32(bk, a[mi][4 * t + c], acc[h][mi], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int RP, int MI, int NR>
__device__ __forceinline__ void l_tile(floatx4 (&lt)[MI], const float (&a)[MI][RP / 4],
                                       const float4 (&pre)[l_lookahead<RP>()],
                                       float (&ring)[NR > 0 ? NR : 1][RP / 16], const float* tile,
                                       int jb, int q, int l16) {
  floatx4 acc[l_chains<MI>()][MI];
  l_tile_acc<RP, MI, NR>(acc, a, pre, ring, tile, jb, q, l16);
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
    lt[mi] = acc[0][mi];
#pragma unroll
    for (int h = 1; h < l_chains<MI>(); ++h) lt[mi] += acc[h][mi];
  }
}

// srcB operands of the second product for k-slice v of j-block jb: P[jb*16 + 4q + v][16 cb + l16].
template <int RP>
__device__ __forceinline__ void zb_read(float (&bb)[RP / 16], const float* tile, int jb, int v,
                                        int q, int l16) {
  const float* b2 = &tile[(jb * 16 + 4 * q + v) * (RP + 4) + l16];
#pragma unroll
  for (int cb = 0; cb < RP / 16; ++cb) bb[cb] = b2[16 * cb];
}

// Which 16 x 4 slices (mi, v) of the rectified tile z = max(0, L) hold a positive entry: bit
// 4 mi + v of the wave-uniform result.
template <int MI>
__device__ __forceinline__ unsigned live_slices(const floatx4 (&z)[MI]) {
  unsigned m = 0;
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int v = 0; v < 4; ++v)
      if (__any(z[mi][v] > 0.f)) m |= 1u << (4 * mi + v);
  return m;
}

// Y[i][c] += sum_j z[i][j] P[j][c] for one 16-row j-block, z = max(0, L) >= 0: srcA = z (the
// rectified L^T accumulator, register v <-> k-slice 4q + v), srcB from LDS.  A 16 x 4 slice
// (mi, v) of z is one srcA operand; it contributes only if one of its entries is positive (bit
// 4 mi + v of `live`), so the MFMAs of zero slices are skipped (S-hat is sparse).  `ring`
// arrives holding the srcB operands of the first NR slices (read during the first product);
// with NR = 2, slice v + 2 is read into the slot of slice v once that slice's MFMAs are issued.
// Returns the number of slices that ran.
template <int RP, int MI, int NR>
__device__ __forceinline__ int zb_tile(floatx4 (&y)[MI][RP / 16], const floatx4 (&z)[MI],
                                       unsigned live, float (&ring)[NR][RP / 16],
                                       const float* tile, int jb, int q, int l16) {
  static_assert(NR == 2 || NR == 4, "ring depth");
  constexpr int CB = RP / 16;
  // with fewer than 4 column blocks consecutive MFMAs of one row block would depend on each
  // other, so there the row blocks are interleaved and a slice runs for all of them
  constexpr bool PER_MI = CB >= 4;
  int ran = 0;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int slot = NR == 4 ? v : (v & 1);
    if constexpr (PER_MI) {
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) {
        if (live & (1u << (4 * mi + v))) {
#pragma unroll
          for (int cb = 0; cb < CB; ++cb)
            y[mi][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(z[mi][v], ring[slot][cb], y[mi][cb], 0, 0, 0);
          ++ran;
        }
      }
    } else {
      unsigned any = 0;
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) any |= live & (1u << (4 * mi + v));
      if (any) {
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
          for (int mi = 0; mi < MI; ++mi)
            y[mi][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(z[mi][v], ring[slot][cb], y[mi][cb], 0, 0, 0);
        ran += MI;
      }
    }
    if constexpr (NR == 2) {
      if (v + 2 < 4) zb_read<RP>(ring[v & 1], tile, jb, v + 2, q, l16);
    }
  }
  return ran;
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

}  // namespace nmd
