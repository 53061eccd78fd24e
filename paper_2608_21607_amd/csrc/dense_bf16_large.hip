// The both-products split-bf16 contraction at r_p = 256 and 512 in the 16 x 16 x 32 form (helpers
// in dense_bf16.h), with a single row-major split panel read both ways.  Compiled with the
// default register allocation: at 512 the single wave per SIMD keeps its output tiles in
// accumulation registers.

#include "dense_bf16.h"
#include "nmd_internal.h"

namespace nmd {
namespace bx {

// ---------------------------------------------------------------------------------------------
// r_p = 256 (two waves per SIMD) and 512 (one wave per SIMD), 16 rows of X per wave.  Only the
// row-major split panel is kept: the second product reads its operand, eight consecutive panel
// rows of one column per lane, out of the same LDS rows with the transposing LDS read of gfx950
// (ds_read_b64_tr_b16), so a panel element costs 4 bytes of traffic (bf16 hi and lo), as in the
// fp32 kernel.  A 32-row block takes r_p / 256 stages of 32 KB (its 256-column halves at 512); a
// ring of four slots holds the block being computed and the next one, loaded while the current
// one runs.  Each stage loads exactly 32 chunks of 1 KB (8 per wave at 512, 4 at 256; rows past
// the panel read a clamped row, and their rectified values are masked to zero), so the per-wave
// load count per stage is fixed for the vmcnt waits.
//
// Stage row layout (1 KB: 256 columns of one panel row): 32 hi chunks then 32 lo chunks of
// 8 columns, chunk c of row r stored at c ^ f(r), f(r) = 2 (r & 7) + ((r >> 3) & 1).  Both reads
// then touch 16 distinct 16-byte bank groups in each 256 bytes: the first product's (rows 0..15
// of one chunk) because f is a permutation of 0..15, the transposing read's (per 32 lanes, rows
// 8p..8p+7, two adjacent chunks) because f(r) >> 1 = r & 7 takes eight values there.  Measured,
// this halves the LDS bank-conflict cycles of a three-bit swizzle (2.67 to 1.33 per LDS
// instruction) at the same speed or slightly better.

template <int RP_>
struct CfgL {
  static constexpr int RP = RP_;
  static constexpr int WAVES = RP >= 512 ? 4 : 8;    // one wave per SIMD at 512, two at 256
  static constexpr int ROWS = 16 * WAVES;             // rows of X per workgroup
  static constexpr int H = RP / 256;                  // 256-column stages per 32-row block
  static constexpr int SLOT = 8192;                   // floats per stage (32 KB)
  static constexpr int LPW = SLOT / 256 / WAVES;      // 1 KB direct loads per wave per stage
  static constexpr int KC = RP / 32;                  // 32-wide k chunks
  static constexpr int CB = RP / 16;                  // 16-column blocks of Y
  static_assert(RP == 256 || RP == 512, "rank");
};

__device__ __forceinline__ int swz_l(int r) { return ((r & 7) << 1) | ((r >> 3) & 1); }

// Workgroup barrier for the staged ring: this wave's direct loads up to the last N have landed
// in LDS (vmcnt <= N) and its LDS reads are done (lgkmcnt 0), then s_barrier.  Unlike
// __syncthreads, no release fence, which would also wait for the N loads still in flight.  The
// empty asm statements keep the compiler from moving memory accesses across the barrier.
template <int N>
__device__ __forceinline__ void ring_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4));
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Row-major split panel: per row, for each 256-column half, the hi chunks of its 32 groups of 8
// columns, then their lo chunks.
template <int RP>
__global__ __launch_bounds__(256) void bxl_split_kernel(const float* __restrict__ P, int64_t blk,
                                                        u32x4* __restrict__ rowm) {
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= blk * (RP / 8)) return;
  const int64_t row = gid / (RP / 8);
  const int g = (int)(gid - row * (RP / 8));
  const float4 a = *reinterpret_cast<const float4*>(P + row * RP + 8 * g);
  const float4 b = *reinterpret_cast<const float4*>(P + row * RP + 8 * g + 4);
  const float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  u32x4 hi, lo;
  split8(x, hi, lo);
  u32x4* dst = rowm + row * (RP / 4) + (g >> 5) * 64 + (g & 31);
  dst[0] = hi;
  dst[32] = lo;
}

// Issue the direct loads of half h (columns 256 h ..) of the 32-row block at panel row j0 into
// `slot`: row r of the block goes to slot row r, its chunk c to position c ^ f(r).
template <int RP>
__device__ __forceinline__ void stage_l(float* slot, int h, const float* __restrict__ rowm,
                                        int64_t j0, int64_t blk, int wave, int lane) {
  using C = CfgL<RP>;
#pragma unroll
  for (int u = 0; u < C::LPW; ++u) {
    const int r = wave + C::WAVES * u;          // row of the block (0..31)
    int64_t j = j0 + r;
    j = j < blk ? j : blk - 1;                  // rows past the panel: any valid row (masked)
    const int c = lane ^ swz_l(r);              // chunk stored at position `lane`
    __builtin_amdgcn_global_load_lds((glb_void*)(rowm + j * C::RP + 256 * h + 4 * c),
                                     (lds_void*)(slot + 256 * r), 16, 0, 0);
  }
}

// First-product chunks of one k-half (a stage slot) into the six chains: a0 for panel rows
// 0..15 of the block, a1 for rows 16..31 (hi x hi, hi x lo, lo x hi each).
template <int RP>
__device__ __forceinline__ void gemm1_half(floatx4 (&a0)[3], floatx4 (&a1)[3], const float* slot,
                                           int half, const u32x4 (&xh)[RP / 32],
                                           const u32x4 (&xl)[RP / 32], int q, int l16) {
  const u32x4* r0 = reinterpret_cast<const u32x4*>(slot + 256 * l16);
  const u32x4* r1 = reinterpret_cast<const u32x4*>(slot + 256 * (16 + l16));
  const int sw = swz_l(l16);  // rows l16 and 16 + l16 share f
  constexpr int LA = 2;
  u32x4 h0[8], o0[8], h1[8], o1[8];
#pragma unroll
  for (int t = 0; t < LA; ++t) {
    const int c = (4 * t + q) ^ sw;
    h0[t] = r0[c];
    o0[t] = r0[32 + c];
    h1[t] = r1[c];
    o1[t] = r1[32 + c];
  }
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    if (t + LA < 8) {
      const int c = (4 * (t + LA) + q) ^ sw;
      h0[t + LA] = r0[c];
      o0[t + LA] = r0[32 + c];
      h1[t + LA] = r1[c];
      o1[t + LA] = r1[32 + c];
    }
    const int k = 8 * half + t;
    a0[0] = mfma(h0[t], xh[k], a0[0]);
    a1[0] = mfma(h1[t], xh[k], a1[0]);
    a0[1] = mfma(h0[t], xl[k], a0[1]);
    a1[1] = mfma(h1[t], xl[k], a1[1]);
    a0[2] = mfma(o0[t], xh[k], a0[2]);
    a1[2] = mfma(o1[t], xh[k], a1[2]);
    __builtin_amdgcn_sched_barrier(0);
  }
}

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;

// One transposing LDS read (ds_read_b64_tr_b16): in each group of 16 lanes, lane i receives, as
// its element e, element i & 3 of the 8 bytes that lane (i >> 2) + 4 e of the group points at.
// (The compiler waits for every direct load in flight before the first of these reads after
// one; measured, that costs less than hand-placed waits around inline assembly.)
__device__ __forceinline__ uint2 tr16(const char* p) {
  const v4s v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)p);
  return __builtin_bit_cast(uint2, v);
}

// Second-product operand of column block cb (16 columns of the half at `base`): lane (q, l16)
// receives the hi and lo parts of panel rows 4q..4q+3 and 16+4q..16+4q+3 of column 16 cb + l16,
// the k order of zsplit.  So lane 16 q + j points at row 4 q + (j >> 2) (jr), columns
// 16 cb + 4 (j & 3) .. + 3 (jc = j & 3), and a second read 16 rows further.  Four LDS reads.
__device__ __forceinline__ void load_b_tr(u32x4& bh, u32x4& bl, const char* base, int cb,
                                          int jr, int jc, int sw) {
  const int c = (2 * cb + (jc >> 1)) ^ sw;                     // hi chunk of the columns
  const char* pa = base + 1024 * jr + 16 * c + 8 * (jc & 1);
  const uint2 h0 = tr16(pa), h1 = tr16(pa + 16 * 1024);
  const uint2 l0 = tr16(pa + 512), l1 = tr16(pa + 16 * 1024 + 512);
  bh = u32x4{h0.x, h0.y, h1.x, h1.y};
  bl = u32x4{l0.x, l0.y, l1.x, l1.y};
}

// Second product for one column half (a stage slot).
template <int RP>
__device__ __forceinline__ void gemm2_half(floatx4 (&y)[RP / 16], const float* slot, int half,
                                           u32x4 zh, u32x4 zl, int q, int l16) {
  const char* base = reinterpret_cast<const char*>(slot);
  const int jr = 4 * q + (l16 >> 2), jc = l16 & 3, sw = swz_l(jr);
  constexpr int G = 2;
  u32x4 nh[G], nl[G];
#pragma unroll
  for (int g = 0; g < G; ++g) load_b_tr(nh[g], nl[g], base, g, jr, jc, sw);
#pragma unroll
  for (int cb0 = 0; cb0 < 16; cb0 += G) {
    u32x4 ch[G], cl[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      ch[g] = nh[g];
      cl[g] = nl[g];
    }
    if (cb0 + G < 16) {
#pragma unroll
      for (int g = 0; g < G; ++g) load_b_tr(nh[g], nl[g], base, cb0 + G + g, jr, jc, sw);
    }
#pragma unroll
    for (int g = 0; g < G; ++g) y[16 * half + cb0 + g] = mfma(zh, ch[g], y[16 * half + cb0 + g]);
#pragma unroll
    for (int g = 0; g < G; ++g) y[16 * half + cb0 + g] = mfma(zh, cl[g], y[16 * half + cb0 + g]);
#pragma unroll
    for (int g = 0; g < G; ++g) y[16 * half + cb0 + g] = mfma(zl, ch[g], y[16 * half + cb0 + g]);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int RP>
__global__ __launch_bounds__(64 * CfgL<RP>::WAVES) void bxl_kernel(
    const float* __restrict__ X, int64_t rows, const float* __restrict__ rowm, int64_t blk,
    float* __restrict__ Ypart, int64_t y_stride, int nsplit, int64_t row_tiles, float sgn,
    unsigned long long* __restrict__ live_slices) {
  using C = CfgL<RP>;
  __shared__ __attribute__((aligned(16))) float ring[4 * C::SLOT];
  static_assert(C::H <= 2, "the ring holds two blocks of two stages");
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int q = lane >> 4, l16 = lane & 15;

  const int64_t logical = xcd_logical(blockIdx.x, (int64_t)gridDim.x);
  const int split = (int)(logical / row_tiles);
  const int64_t rt = logical - (int64_t)split * row_tiles;
  const int64_t jb0 = pair_start(split, nsplit, blk);
  const int64_t jb1 = pair_start(split + 1, nsplit, blk);
  const int64_t row0 = rt * C::ROWS + (int64_t)wave * 16;

  u32x4 xh[C::KC], xl[C::KC];
  load_x<RP>(xh, xl, X, rows, row0, q, l16);
  floatx4 y[C::CB];
  {
    // zero the output tiles with an MFMA of zero operands: their loop-carried values then start
    // in accumulation registers, and the skipped second products cost no register copies
    const u32x4 z0 = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int cb = 0; cb < C::CB; ++cb) y[cb] = mfma(z0, z0, floatx4{0.f, 0.f, 0.f, 0.f});
  }

  const int64_t nblk = (jb1 - jb0 + 31) / 32;
  unsigned ran = 0;
  unsigned pos = 0;  // positive entries of max(0, L) this lane saw
  if (nblk > 0) {
    // stage h of block b goes to slot (H b + h) mod 4: at H = 2 the ring holds this block and
    // the next, at H = 1 the block and the next three slots
#pragma unroll
    for (int h = 0; h < C::H; ++h) stage_l<RP>(ring + h * C::SLOT, h, rowm, jb0, blk, wave, lane);
    for (int64_t b = 0; b < nblk; ++b) {
      const int64_t j0 = jb0 + 32 * b;
      const float* s0 = ring + (int)((C::H * b) & 3) * C::SLOT;
      const float* s1 = C::H > 1 ? s0 + C::SLOT : s0;
      // stage 0 of this block landed for every wave; every wave is done with the previous block
      ring_barrier<(C::H - 1) * C::LPW>();
      const bool more = b + 1 < nblk;
      if (more) {
#pragma unroll
        for (int h = 0; h < C::H; ++h)
          stage_l<RP>(ring + (int)((C::H * (b + 1) + h) & 3) * C::SLOT, h, rowm, j0 + 32, blk,
                      wave, lane);
      }
      floatx4 a0[3], a1[3];
#pragma unroll
      for (int h = 0; h < 3; ++h) a0[h] = a1[h] = floatx4{0.f, 0.f, 0.f, 0.f};
      gemm1_half<RP>(a0, a1, s0, 0, xh, xl, q, l16);
      if constexpr (C::H > 1) {
        // stage 1 of this block landed for every wave (the next block's loads stay in flight)
        if (more) ring_barrier<C::H * C::LPW>();
        else ring_barrier<0>();
        gemm1_half<RP>(a0, a1, s1, 1, xh, xl, q, l16);
      }
      const floatx4 l0 = a0[0] + (a0[1] + a0[2]);
      const floatx4 l1 = a1[0] + (a1[1] + a1[2]);
      // panel rows of this block inside the range (only values below 32 mask anything)
      const int valid = (int)(jb1 - j0 < 32 ? jb1 - j0 : 32);
      floatx4 m0, m1;
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        m0[v] = 4 * q + v < valid ? l0[v] : 0.f;
        m1[v] = 16 + 4 * q + v < valid ? l1[v] : 0.f;
        pos += (m0[v] > 0.f ? 1u : 0u) + (m1[v] > 0.f ? 1u : 0u);
      }
      u32x4 zh, zl;
      if (zsplit(m0, m1, zh, zl)) {
        ++ran;
        gemm2_half<RP>(y, s0, 0, zh, zl, q, l16);
        if constexpr (C::H > 1) gemm2_half<RP>(y, s1, 1, zh, zl, q, l16);
      }
    }
  }

  float* Y = Ypart + (int64_t)split * y_stride;
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int64_t row = row0 + 4 * q + v;
    if (row < rows) {
#pragma unroll
      for (int cb = 0; cb < C::CB; ++cb) Y[row * C::RP + 16 * cb + l16] = sgn * y[cb][v];
    }
  }
  // a live 16 x 32 tile counts as its eight 16 x 4 slices of max(0, L); [1] counts the positive
  // entries (rows of X past `rows` are zero and add none)
  if (live_slices) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) pos += __shfl_xor(pos, off, 64);
    if (lane == 0 && ran) atomicAdd(live_slices, 8ull * ran);
    if (lane == 0 && pos) atomicAdd(live_slices + 1, (unsigned long long)pos);
  }
}

}  // namespace bx

// r_p = 512: staged four-slot form.
template <int RP>
static hipError_t bxl_launch(const float* X, int64_t rows, const float* P, int64_t blk,
                             float* work, float* Ypart, int64_t y_stride, int nsplit, float sgn,
                             unsigned long long* live, hipStream_t st) {
  using C = bx::CfgL<RP>;
  const int64_t threads = blk * (RP / 8);
  hipLaunchKernelGGL(bx::bxl_split_kernel<RP>, dim3((unsigned)((threads + 255) / 256)), dim3(256),
                     0, st, P, blk, reinterpret_cast<bx::u32x4*>(work));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t row_tiles = (rows + C::ROWS - 1) / C::ROWS;
  const int64_t total = row_tiles * nsplit;
  if (total <= 0) return hipSuccess;
  if (total > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(bx::bxl_kernel<RP>, dim3((unsigned)total), dim3(64 * C::WAVES), 0, st, X,
                     rows, work, blk, Ypart, y_stride, nsplit, row_tiles, sgn, live);
  return hipGetLastError();
}

hipError_t launch_bf16x3_staged(const float* X, int64_t rows, const float* P, int64_t blk, int rp,
                                float* work, float* Ypart, int64_t y_stride, int nsplit,
                                float sgn, unsigned long long* live, hipStream_t st) {
  switch (rp) {
    case 256: return bxl_launch<256>(X, rows, P, blk, work, Ypart, y_stride, nsplit, sgn, live, st);
    case 512: return bxl_launch<512>(X, rows, P, blk, work, Ypart, y_stride, nsplit, sgn, live, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace nmd
