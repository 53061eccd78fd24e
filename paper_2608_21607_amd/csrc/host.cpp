// libnmd host side: the C ABI declared in include/nmd.h.
//
// Owns the context (problem sizes, block partition, copies of S arranged per block, device
// workspaces, momentum buffers, sweep counter), validates every argument before any device
// work, builds the per-sweep block order, and enqueues the kernels of each update on the
// caller's stream.  Nothing here computes the method's arithmetic; the kernels do.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstddef>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/nmd.h"
#include "nmd_internal.h"


using nmd::Item;
using nmd::Split;
using nmd::balanced_bounds;
using nmd::make_schedule;

namespace {

thread_local std::string g_create_error;

constexpr int kMaxSplits = 16;     // partial outputs of the dense kernel
constexpr int64_t kSplitRows = 8192;  // at most this many panel rows per fp32 accumulation
constexpr int64_t kTargetWgs = 2048;  // dense workgroups wanted per launch (256 CUs)
constexpr int64_t kWgFixedRows = 32;  // per-workgroup set-up and write-back, in panel rows
constexpr int kObjSubMax = 16;        // sub-splits of a column block in the objective
// Steps one call may enqueue: the device status word keeps step_id * 8 + flag in an int.
constexpr int64_t kMaxStepsPerCall = int64_t{1} << 27;

enum { K_DENSE = 0, K_SPARSE = 1, K_FACTOR = 2, K_APPLY = 3, K_JOIN = 4, K_COUNT = 5 };

// The arrangement of S for one factor (ingest.h) and its device copies.
struct Side : nmd::SideHost {
  int32_t* d_idx = nullptr;
  float* d_val = nullptr;
  Item* d_items = nullptr;
  Split* d_splits = nullptr;
  int64_t* d_rowptr = nullptr;
  int64_t* d_bounds = nullptr;
};

struct TimerRec {
  hipEvent_t a, b;
  int kind;
  double flops, bytes;
};

}  // namespace

struct nmd_ctx {
  int64_t m = 0, n = 0;
  int32_t r = 0, rp = 0;
  int32_t block_m = 0, block_n = 0;
  uint64_t seed = 0;
  nmd_options opt{};
  std::vector<int64_t> rb, cb;  // row and column block bounds
  int64_t t = 0;
  float eta0 = 1.0f;           // step size at creation (the safeguard may lower opt.eta)
  int64_t rejected = 0;        // sweeps undone by the step-size safeguard
  int last_fail_step = -1;     // step id of the last step the device rejected
  std::string err;

  bool has_S = false;
  int64_t nnz = 0;
  double s_norm = 0.0;
  Side ws, hs;  // W side (column blocks), H side (row blocks)
  std::vector<int64_t> nnz_col_blocks, nnz_row_blocks;

  // device state
  bool dev_ready = false;
  bool sparse_uploaded = false;
  int device = -1;
  // Factors (padded, B = H^T) and momenta: the current buffers and a second one of each.  A
  // step reads the current factor and momentum and writes the other pair, which then becomes
  // current, so a step the device rejects leaves the state of the last completed step intact.
  float *A = nullptr, *B = nullptr, *VA = nullptr, *VB = nullptr;
  float *A2 = nullptr, *B2 = nullptr, *VA2 = nullptr, *VB2 = nullptr;
  std::vector<std::pair<int, bool>> enqueued;  // (step id, W-step) of the call's steps, in order
  float* Ypart = nullptr;
  float* Pbx = nullptr;  // split-bf16 panel copies (NMD_FLAG_SPLIT_BF16 at r_p = 16..512)
  int64_t ypart_floats = 0;
  float* scratch = nullptr;
  int64_t scratch_floats = 0;

  double *G = nullptr, *Gwork = nullptr, *Gpart = nullptr;
  double* Gneg[nmd::kSolveBatch] = {};  // -G^-1 of each step of the current run (in Gwork)
  int gram_chunks_max = 64;
  double* objpart = nullptr;
  int64_t objpart_count = 0;
  double* objout = nullptr;
  // per-sweep objectives (sums of squares) of the last sweep call: [0] before its first sweep
  double* fhist = nullptr;
  int64_t fhist_cap = 0, fcount = 0;
  float *SA = nullptr, *SB = nullptr;  // the factors before the current sweep (safeguard)
  int* status = nullptr;
  unsigned long long* g2 = nullptr;  // [0] S-hat slices whose second product ran whole,
                                     // [1] S-hat entries taken through gathered slices
  int64_t g2_total = 0;              // slices examined (host count)
  int64_t dense_slots = 0;           // dense workgroups resident at once (CUs x per CU)
  hipStream_t side = nullptr;     // Gram and inverse run here, beside the contraction
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  hipStream_t corr = nullptr;     // the sparse correction runs here, beside the contraction
  hipEvent_t ev_cfork = nullptr, ev_cjoin = nullptr;
  float* Ysp = nullptr;           // its output there (max(m, n) rows x rp; r_p >= 320, fp32)
  int* h_status = nullptr;   // pinned
  double* h_obj = nullptr;   // pinned

  // timing
  std::vector<TimerRec> pending;
  std::vector<hipEvent_t> event_pool;
  double t_ms[K_COUNT] = {};
  int64_t t_launch[K_COUNT] = {};
  double t_flops[K_COUNT] = {};
  double t_bytes[K_COUNT] = {};
};

namespace {

int fail(nmd_ctx* c, int code, const char* fmt, ...) __attribute__((format(printf, 3, 4)));
int fail(nmd_ctx* c, int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c)
    c->err = buf;
  else
    g_create_error = buf;
  return code;
}

#define HIP_TRY(ctx, expr)                                                                  \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return fail(ctx, NMD_EDEVICE, "%s failed: %s", #expr, hipGetErrorString(e_));         \
  } while (0)

template <class T>
hipError_t dalloc(T** p, int64_t count) {
  *p = nullptr;
  if (count <= 0) count = 1;
  return hipMalloc((void**)p, (size_t)count * sizeof(T));
}

template <class T>
void dfree(T*& p) {
  if (p) (void)hipFree(p);
  p = nullptr;
}

void free_sparse_device(nmd_ctx* c) {
  for (Side* sd : {&c->ws, &c->hs}) {
    dfree(sd->d_idx);
    dfree(sd->d_val);
    dfree(sd->d_items);
    dfree(sd->d_splits);
    dfree(sd->d_rowptr);
    dfree(sd->d_bounds);
  }
  dfree(c->scratch);
  dfree(c->objpart);
  c->sparse_uploaded = false;
}

void free_device(nmd_ctx* c) {
  free_sparse_device(c);
  dfree(c->A);
  dfree(c->B);
  dfree(c->VA);
  dfree(c->VB);
  dfree(c->A2);
  dfree(c->B2);
  dfree(c->VA2);
  dfree(c->VB2);
  dfree(c->Ypart);
  dfree(c->Pbx);
  dfree(c->G);
  dfree(c->Gwork);
  dfree(c->Gpart);
  dfree(c->objout);
  dfree(c->fhist);
  c->fhist_cap = c->fcount = 0;
  dfree(c->SA);
  dfree(c->SB);
  dfree(c->status);
  dfree(c->g2);
  if (c->ev_fork) (void)hipEventDestroy(c->ev_fork);
  if (c->ev_join) (void)hipEventDestroy(c->ev_join);
  if (c->side) (void)hipStreamDestroy(c->side);
  c->ev_fork = c->ev_join = nullptr;
  c->side = nullptr;
  if (c->ev_cfork) (void)hipEventDestroy(c->ev_cfork);
  if (c->ev_cjoin) (void)hipEventDestroy(c->ev_cjoin);
  if (c->corr) (void)hipStreamDestroy(c->corr);
  c->ev_cfork = c->ev_cjoin = nullptr;
  c->corr = nullptr;
  dfree(c->Ysp);
  if (c->h_status) (void)hipHostFree(c->h_status);
  if (c->h_obj) (void)hipHostFree(c->h_obj);
  c->h_status = nullptr;
  c->h_obj = nullptr;
  for (auto& rec : c->pending) {
    (void)hipEventDestroy(rec.a);
    (void)hipEventDestroy(rec.b);
  }
  c->pending.clear();
  for (hipEvent_t e : c->event_pool) (void)hipEventDestroy(e);
  c->event_pool.clear();
  c->dev_ready = false;
}

// Number of disjoint panel ranges (partial outputs) of one dense launch.  At least enough for
// kTargetWgs workgroups and for at most kSplitRows panel rows per fp32 accumulation; beyond that
// the count that wastes the least of the last round of workgroups on `slots` concurrent
// workgroups (CUs x workgroups per CU), each workgroup costing its panel rows plus a fixed
// equivalent of kWgFixedRows for loading its rows of X and writing its output.
int64_t nsplit_for(int64_t rows, int64_t blk, int rp, int64_t slots) {
  const int64_t rw = nmd::dense_rows_per_wg(rp);
  const int64_t tiles = (rows + rw - 1) / rw;
  const int64_t cap = std::max<int64_t>(1, std::min<int64_t>(kMaxSplits, blk / 16));
  int64_t lo = std::max<int64_t>((blk + kSplitRows - 1) / kSplitRows, (kTargetWgs + tiles - 1) / tiles);
  lo = std::max<int64_t>(1, std::min(lo, cap));
  if (slots < 1) return lo;
  int64_t best = lo;
  double best_cost = 0.0;
  for (int64_t s = lo; s <= cap; ++s) {
    const int64_t rounds = (tiles * s + slots - 1) / slots;
    const double cost = (double)rounds * ((double)blk / (double)s + (double)kWgFixedRows);
    if (s == lo || cost < best_cost * 0.995) {  // a larger count must win by a margin
      best = s;
      best_cost = cost;
    }
  }
  return best;
}

int gram_chunks(int64_t blk) {
  return (int)std::min<int64_t>(64, std::max<int64_t>(1, blk / 256));
}

int ensure_device(nmd_ctx* c) {
  if (!c->dev_ready) {
    int dev = 0;
    HIP_TRY(c, hipGetDevice(&dev));
    hipDeviceProp_t prop;
    HIP_TRY(c, hipGetDeviceProperties(&prop, dev));
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
      return fail(c, NMD_EDEVICE, "device %d is %s; this library is built for gfx950", dev,
                  prop.gcnArchName);
    c->device = dev;
    const int64_t rp = c->rp;
    int per_cu = 0;
    HIP_TRY(c, nmd::dense_wgs_per_cu(c->rp, &per_cu));
    c->dense_slots = (int64_t)prop.multiProcessorCount * std::max(per_cu, 1);
    const int64_t mpad = c->m + 256, npad = c->n + 256;
    if (dalloc(&c->A, mpad * rp) != hipSuccess || dalloc(&c->B, npad * rp) != hipSuccess ||
        dalloc(&c->VA, mpad * rp) != hipSuccess || dalloc(&c->VB, npad * rp) != hipSuccess ||
        dalloc(&c->A2, mpad * rp) != hipSuccess || dalloc(&c->B2, npad * rp) != hipSuccess ||
        dalloc(&c->VA2, mpad * rp) != hipSuccess || dalloc(&c->VB2, npad * rp) != hipSuccess ||
        dalloc(&c->G, nmd::kSolveBatch * rp * rp) != hipSuccess ||
        dalloc(&c->Gwork, nmd::kSolveBatch * nmd::chol_work_doubles((int)rp)) != hipSuccess ||
        dalloc(&c->Gpart, (int64_t)c->gram_chunks_max * rp * rp) != hipSuccess ||
        dalloc(&c->objout, 8) != hipSuccess || dalloc(&c->status, 2) != hipSuccess ||
        dalloc(&c->g2, 2) != hipSuccess) {
      free_device(c);
      return fail(c, NMD_ENOMEM, "device allocation of the factor workspaces failed");
    }
    // Partial outputs: the largest (splits x rows) over W-steps, H-steps and full half-sweeps.
    int64_t need = 0;
    for (size_t k = 0; k + 1 < c->cb.size(); ++k) {
      const int64_t blk = c->cb[k + 1] - c->cb[k];
      need = std::max(need, nsplit_for(c->m, blk, c->rp, c->dense_slots) * c->m);
    }
    for (size_t k = 0; k + 1 < c->rb.size(); ++k) {
      const int64_t blk = c->rb[k + 1] - c->rb[k];
      need = std::max(need, nsplit_for(c->n, blk, c->rp, c->dense_slots) * c->n);
    }
    need = std::max(need, nsplit_for(c->m, c->n, c->rp, c->dense_slots) * c->m);
    need = std::max(need, nsplit_for(c->n, c->m, c->rp, c->dense_slots) * c->n);
    c->ypart_floats = need * rp;
    // the split-bf16 option covers the padded ranks the bf16x3 kernels support
    const bool bx = (c->opt.flags & NMD_FLAG_SPLIT_BF16) && nmd::bf16x3_rank(rp);
    if (dalloc(&c->Ypart, c->ypart_floats) != hipSuccess ||
        (rp >= 320 && !bx && dalloc(&c->Ysp, std::max(c->m, c->n) * rp) != hipSuccess) ||
        (bx && dalloc(&c->Pbx, nmd::bf16x3_work_floats(std::max(c->m, c->n), rp)) != hipSuccess)) {
      free_device(c);
      return fail(c, NMD_ENOMEM, "device allocation of %lld partial-output floats failed",
                  (long long)c->ypart_floats);
    }
    if (hipHostMalloc((void**)&c->h_status, 2 * sizeof(int)) != hipSuccess ||
        hipHostMalloc((void**)&c->h_obj, 8 * sizeof(double)) != hipSuccess) {
      free_device(c);
      return fail(c, NMD_ENOMEM, "pinned host allocation failed");
    }
    for (float* p : {c->VA, c->VA2, c->A, c->A2})
      HIP_TRY(c, hipMemset(p, 0, (size_t)mpad * rp * sizeof(float)));
    for (float* p : {c->VB, c->VB2, c->B, c->B2})
      HIP_TRY(c, hipMemset(p, 0, (size_t)npad * rp * sizeof(float)));
    // default priority on purpose: every stream of the library runs at the same priority
    if (hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&c->ev_fork, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&c->ev_join, hipEventDisableTiming) != hipSuccess ||
        hipStreamCreateWithFlags(&c->corr, hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&c->ev_cfork, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&c->ev_cjoin, hipEventDisableTiming) != hipSuccess) {
      free_device(c);
      return fail(c, NMD_EDEVICE, "creating the side streams or their events failed");
    }
    HIP_TRY(c, hipMemset(c->status, 0, sizeof(int)));
    HIP_TRY(c, hipMemset(c->status + 1, 0x7f, sizeof(int)));
    HIP_TRY(c, hipMemset(c->g2, 0, 2 * sizeof(unsigned long long)));
    HIP_TRY(c, hipDeviceSynchronize());
    c->dev_ready = true;
  } else {
    HIP_TRY(c, hipSetDevice(c->device));
  }
  if (c->has_S && !c->sparse_uploaded) {
    for (Side* sd : {&c->ws, &c->hs}) {
      const int64_t nz = (int64_t)sd->idx.size();
      if (dalloc(&sd->d_idx, nz) != hipSuccess || dalloc(&sd->d_val, nz) != hipSuccess ||
          dalloc(&sd->d_items, (int64_t)sd->items.size()) != hipSuccess ||
          dalloc(&sd->d_splits, (int64_t)sd->splits.size()) != hipSuccess ||
          dalloc(&sd->d_rowptr, (int64_t)sd->rowptr.size()) != hipSuccess ||
          dalloc(&sd->d_bounds, (int64_t)sd->bounds.size()) != hipSuccess) {
        free_sparse_device(c);
        return fail(c, NMD_ENOMEM, "device allocation of the sparse structures failed");
      }
      HIP_TRY(c, hipMemcpy(sd->d_idx, sd->idx.data(), nz * sizeof(int32_t), hipMemcpyHostToDevice));
      HIP_TRY(c, hipMemcpy(sd->d_val, sd->val.data(), nz * sizeof(float), hipMemcpyHostToDevice));
      if (!sd->items.empty())
        HIP_TRY(c, hipMemcpy(sd->d_items, sd->items.data(), sd->items.size() * sizeof(Item),
                             hipMemcpyHostToDevice));
      if (!sd->splits.empty())
        HIP_TRY(c, hipMemcpy(sd->d_splits, sd->splits.data(), sd->splits.size() * sizeof(Split),
                             hipMemcpyHostToDevice));
      HIP_TRY(c, hipMemcpy(sd->d_rowptr, sd->rowptr.data(), sd->rowptr.size() * sizeof(int64_t),
                           hipMemcpyHostToDevice));
      HIP_TRY(c, hipMemcpy(sd->d_bounds, sd->bounds.data(), sd->bounds.size() * sizeof(int64_t),
                           hipMemcpyHostToDevice));
    }
    c->scratch_floats = std::max<int64_t>(1, std::max(c->ws.max_slots, c->hs.max_slots)) * c->rp;
    // objective partials: one per (row tile, column block, sub-split)
    c->objpart_count = 5 * (int64_t)nmd::dense_max_wgs(c->m, c->rp, 1) * c->ws.nblk() * kObjSubMax + 1;
    if (dalloc(&c->scratch, c->scratch_floats) != hipSuccess ||
        dalloc(&c->objpart, c->objpart_count) != hipSuccess) {
      free_sparse_device(c);
      return fail(c, NMD_ENOMEM, "device allocation of the sparse scratch failed");
    }
    c->sparse_uploaded = true;
  }
  return NMD_OK;
}

// ---------------------------------------------------------------------------- timing --
hipEvent_t take_event(nmd_ctx* c) {
  if (!c->event_pool.empty()) {
    hipEvent_t e = c->event_pool.back();
    c->event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

struct Scope {
  nmd_ctx* c;
  hipStream_t st;
  TimerRec rec{};
  bool on;
  Scope(nmd_ctx* c_, hipStream_t st_, int kind, double flops, double bytes)
      : c(c_), st(st_), on((c_->opt.flags & NMD_FLAG_TIMING) != 0) {
    if (!on) return;
    rec.a = take_event(c);
    rec.b = take_event(c);
    rec.kind = kind;
    rec.flops = flops;
    rec.bytes = bytes;
    if (!rec.a || !rec.b) {
      on = false;
      return;
    }
    (void)hipEventRecord(rec.a, st);
  }
  ~Scope() {
    if (!on) return;
    (void)hipEventRecord(rec.b, st);
    c->pending.push_back(rec);
  }
};

int collect_timing(nmd_ctx* c) {
  for (auto& rec : c->pending) {
    HIP_TRY(c, hipEventSynchronize(rec.b));
    float ms = 0.f;
    HIP_TRY(c, hipEventElapsedTime(&ms, rec.a, rec.b));
    c->t_ms[rec.kind] += ms;
    c->t_launch[rec.kind] += 1;
    c->t_flops[rec.kind] += rec.flops;
    c->t_bytes[rec.kind] += rec.bytes;
    c->event_pool.push_back(rec.a);
    c->event_pool.push_back(rec.b);
  }
  c->pending.clear();
  return NMD_OK;
}

// ---------------------------------------------------------------------- one update step --
// wstep: update A = W from column block `block` (all column blocks if block < 0); otherwise
// update B = H^T from row block `block` (all row blocks if block < 0).
// The other buffers of one side's factor and momentum become current.
void swap_side(nmd_ctx* c, bool wside) {
  if (wside) {
    std::swap(c->A, c->A2);
    std::swap(c->VA, c->VA2);
  } else {
    std::swap(c->B, c->B2);
    std::swap(c->VB, c->VB2);
  }
}

// The Gram matrices of a run of consecutive steps of one side and their -G^-1: they depend only
// on the panel rows of each step's block, and the run's steps change only the other factor, so
// the whole run's solves are formed in one set of launches on the side stream while the first
// step's contraction runs on the caller's stream; every apply of the run waits for them.
// blocks[i] < 0 (deterministic mode) takes every block of the side as one step.
int factor_run(nmd_ctx* c, bool wstep, const int32_t* blocks, int n, int first_step_id,
               hipStream_t st) {
  const Side& sd = wstep ? c->ws : c->hs;
  const float* P = wstep ? c->B : c->A;
  nmd::SolveBatch sb{};
  sb.n = n;
  double flops = 0.0;
  int64_t blk_max = 0;
  for (int b = 0; b < n; ++b) {
    const int32_t block = blocks[b];
    const int64_t j0 = block >= 0 ? sd.bounds[block] : 0;
    const int64_t j1 = block >= 0 ? sd.bounds[block + 1] : sd.other;
    sb.step_id[b] = first_step_id + b;
    sb.j0[b] = j0;
    sb.blk[b] = j1 - j0;
    blk_max = std::max(blk_max, j1 - j0);
    // Gram 2 blk r^2; Cholesky, inverse of the factor and the product M^T M r^3 / 3 each
    flops += 2.0 * (j1 - j0) * (double)c->r * c->r + (double)c->rp * c->rp * c->rp;
  }
  const int nchunks = std::max(1, std::min(gram_chunks(blk_max), c->gram_chunks_max / n));
  HIP_TRY(c, hipEventRecord(c->ev_fork, st));
  HIP_TRY(c, hipStreamWaitEvent(c->side, c->ev_fork, 0));
  {
    Scope sc(c, c->side, K_FACTOR, flops, 0.0);
    HIP_TRY(c, nmd::launch_gram(P, sb, c->r, c->rp, c->Gpart, nchunks, c->G, c->side));
    // one workgroup per matrix (one launch) at the large and the small ranks; one launch per
    // 64-wide block column, then two, in between, where that is faster on its own
    if (c->rp >= 320 || c->rp <= 64)
      HIP_TRY(c, nmd::launch_chol_inverse_fused(c->G, c->Gwork, c->rp, c->status, sb, c->Gneg,
                                                c->side));
    else
      HIP_TRY(c, nmd::launch_chol_inverse(c->G, c->Gwork, c->rp, c->status, sb, c->Gneg, c->side));
  }
  HIP_TRY(c, hipEventRecord(c->ev_join, c->side));
  return NMD_OK;
}

// One update step with the -G^-1 that factor_run formed for it.
int factor_step(nmd_ctx* c, bool wstep, int32_t block, float eta, float gamma, int step_id,
                const double* Gneg, hipStream_t st) {
  Side& sd = wstep ? c->ws : c->hs;
  float* X = wstep ? c->A : c->B;
  const float* P = wstep ? c->B : c->A;
  float* V = wstep ? c->VA : c->VB;
  const int64_t rows = wstep ? c->m : c->n;
  const int64_t j0 = block >= 0 ? sd.bounds[block] : 0;
  const int64_t j1 = block >= 0 ? sd.bounds[block + 1] : sd.other;
  const int64_t blk = j1 - j0;
  const int rp = c->rp;
  const float* PJ = P + j0 * rp;

  const int64_t ns = nsplit_for(rows, blk, rp, c->dense_slots);
  const int64_t y_stride = rows * rp;
  if (ns * y_stride > c->ypart_floats)
    return fail(c, NMD_EDEVICE, "internal: partial-output buffer too small");
  // Where the contraction runs one matrix-core wave per SIMD (r_p >= 320, fp32), the sparse
  // correction runs beside it, on its own stream, into its own buffer: it is bound by memory
  // and needs no LDS, so its workgroups fill the register and wave slots the contraction leaves
  // on every CU (co-occurrence sweep 627 -> 608 ms).  At r_p <= 256 the contraction runs two
  // waves per SIMD, and the correction beside it slowed it by more than the correction's own
  // time (graph sweep 202.5 -> 204.5 ms); there it runs after the contraction, on the same
  // stream, added in place to the first partial output.  X and P are final here.
  const bool beside = !c->Pbx && rp >= 320;
  if (beside) {
    HIP_TRY(c, hipEventRecord(c->ev_cfork, st));
    HIP_TRY(c, hipStreamWaitEvent(c->corr, c->ev_cfork, 0));
  }
  {
    // U = Delta_{:J} P_J starts as -max(0, X P_J^T) P_J (eq. updateD off the nonzeros); the
    // second contraction is skipped on the 16 x 4 slices where that rectified tile is zero
    Scope sc(c, st, K_DENSE, 4.0 * rows * (double)blk * c->r, 4.0 * (2.0 * rows + blk) * c->r);
    int64_t jblocks = 0;  // 16-row panel blocks the launch examines
    if (c->Pbx) {  // both products on split bf16: the panel is split once per step
      HIP_TRY(c, nmd::launch_bf16x3(X, rows, PJ, blk, rp, c->Pbx, c->Ypart, y_stride, (int)ns,
                                    -1.0f, c->g2, st));
      for (int s = 0; s < (int)ns; ++s)
        jblocks += 2 * ((nmd::bf16x3_pair_start(s + 1, (int)ns, blk) -
                         nmd::bf16x3_pair_start(s, (int)ns, blk) + 31) / 32);
    } else {
      HIP_TRY(c, nmd::launch_dense(X, rows, PJ, blk, rp, c->Ypart, y_stride, (int)ns, -1.0f,
                                   c->g2, st));
      for (int64_t s = 0; s < ns; ++s) jblocks += ((s + 1) * blk / ns - s * blk / ns + 15) / 16;
    }
    // slices of 16 rows x 4 panel rows examined (those entirely past the last row never run)
    c->g2_total += (rows + 15) / 16 * jblocks * 4;
  }
  // Sparse correction at the nonzeros (eq. updateD there: s - l = (s - min(0, l)) - max(0, l)):
  // beside the contraction into Ysp (zero off the touched rows), else into the first partial.
  hipStream_t cs = beside ? c->corr : st;
  float* Ycorr = beside ? c->Ysp : c->Ypart;
  const int32_t b0 = block >= 0 ? block : 0;
  const int32_t b1 = block >= 0 ? block + 1 : sd.nblk();
  if (beside) HIP_TRY(c, nmd::launch_zero(c->Ysp, rows * rp, cs));
  for (int32_t b = b0; b < b1; ++b) {
    const int64_t ni = sd.item_off[b + 1] - sd.item_off[b];
    const int64_t nsp = sd.split_off[b + 1] - sd.split_off[b];
    const int64_t nz = sd.entry_off[b + 1] - sd.entry_off[b];
    // into the partial output it always adds; into Ysp the first block (every block in the
    // stochastic mode) writes and later ones add
    const int acc = !beside || b > b0 ? 1 : 0;
    // algorithmic bytes: entries (index + value), each touched row of X and of Y (read x,
    // write y, and read y where it adds), each panel row of the block once
    const double bytes = 8.0 * nz + (acc ? 12.0 : 8.0) * (double)ni * c->r + 4.0 * blk * c->r;
    Scope sc(c, cs, K_SPARSE, 4.0 * nz * c->r, bytes);
    HIP_TRY(c, nmd::launch_sparse(sd.d_items + sd.item_off[b], ni, sd.d_idx, sd.d_val, X, P, rp,
                                  Ycorr, c->scratch, acc, cs));
    HIP_TRY(c, nmd::launch_fixup(sd.d_splits + sd.split_off[b], nsp, c->scratch, rp, Ycorr, acc,
                                 cs));
  }
  if (beside) {
    HIP_TRY(c, hipEventRecord(c->ev_cjoin, c->corr));
    HIP_TRY(c, hipStreamWaitEvent(st, c->ev_cjoin, 0));
  }
  {
    // the time the caller's stream waits here for the side stream (zero once it is ahead)
    Scope sc(c, st, K_JOIN, 0.0, 0.0);
    HIP_TRY(c, hipStreamWaitEvent(st, c->ev_join, 0));
  }
  {
    Scope sc(c, st, K_APPLY, 2.0 * rows * (double)rp * rp,
             4.0 * rows * rp * (ns + (beside ? 5 : 4)));
    float* Xout = wstep ? c->A2 : c->B2;
    float* Vout = wstep ? c->VA2 : c->VB2;
    HIP_TRY(c, nmd::launch_apply(c->Ypart, y_stride, (int)ns, beside ? c->Ysp : nullptr, Gneg, X,
                                 V, Xout, Vout, rows, rp, eta, gamma, c->status, step_id, st));
  }
  swap_side(c, wstep);
  c->enqueued.emplace_back(step_id, wstep);
  return NMD_OK;
}

int load_factors(nmd_ctx* c, const float* W, const float* H, hipStream_t st) {
  HIP_TRY(c, nmd::launch_pad_rows(W, c->m, c->r, c->A, c->rp, st));
  HIP_TRY(c, nmd::launch_transpose_in(H, c->r, c->n, c->B, c->rp, st));
  return NMD_OK;
}

int store_factors(nmd_ctx* c, float* W, float* H, hipStream_t st) {
  HIP_TRY(c, nmd::launch_unpad_rows(c->A, c->m, c->rp, W, c->r, st));
  HIP_TRY(c, nmd::launch_transpose_out(c->B, c->rp, c->n, H, c->r, st));
  return NMD_OK;
}

std::string describe_step(nmd_ctx* c, int step_id, int64_t first_sweep, int32_t steps_per) {
  char buf[160];
  if (steps_per <= 0) {
    snprintf(buf, sizeof buf, "step %d", step_id);
  } else {
    snprintf(buf, sizeof buf, "sweep %lld, step %d", (long long)(first_sweep + step_id / steps_per),
             step_id % steps_per);
  }
  (void)c;
  return buf;
}

// Ends a call that ran steps: copies the factors back to W and H and, unless NMD_FLAG_ASYNC is
// set, reports a step the device rejected.  Then the factors stored are those after the last
// completed step: the buffers each side had before the call, swapped once per completed step
// of that side (a rejected step and every step after it wrote only to buffers not current).
int conclude(nmd_ctx* c, float* W, float* H, hipStream_t st, int64_t first_sweep,
             int32_t steps_per) {
  if (c->opt.flags & NMD_FLAG_ASYNC) return store_factors(c, W, H, st);
  HIP_TRY(c, hipMemcpyAsync(c->h_status, c->status, 2 * sizeof(int), hipMemcpyDeviceToHost, st));
  HIP_TRY(c, hipStreamSynchronize(st));
  const int flags = c->h_status[0];
  if (flags == 0) {
    int rc = store_factors(c, W, H, st);
    if (rc) return rc;
    HIP_TRY(c, hipStreamSynchronize(st));
    return NMD_OK;
  }
  const int step = nmd::status_step(c->h_status[1]);
  c->last_fail_step = step;
  for (auto it = c->enqueued.rbegin(); it != c->enqueued.rend(); ++it)
    if (it->first >= step) swap_side(c, it->second);  // undo the steps from the rejected one on
  int rc = store_factors(c, W, H, st);
  if (rc) return rc;
  HIP_TRY(c, hipMemsetAsync(c->status, 0, sizeof(int), st));
  HIP_TRY(c, hipMemsetAsync(c->status + 1, 0x7f, sizeof(int), st));
  HIP_TRY(c, hipStreamSynchronize(st));
  const std::string where = describe_step(c, step, first_sweep, steps_per);
  if (nmd::status_kind(c->h_status[1]) == nmd::STATUS_NOTPD)
    return fail(c, NMD_ENOTPD, "Gram matrix not positive definite at %s; later steps skipped",
                where.c_str());
  return fail(c, NMD_ENONFINITE, "non-finite factor entry produced at %s; later steps skipped",
              where.c_str());
}

int check_ready(nmd_ctx* c, const void* W, const void* H) {
  if (!c) return NMD_EINVAL;
  c->err.clear();
  if (!W || !H) return fail(c, NMD_EINVAL, "W and H must be non-NULL device pointers");
  if (!c->has_S) return fail(c, NMD_ESTATE, "nmd_set_sparse_csr has not been called");
  return NMD_OK;
}

// Enqueues the objective kernel on the current panels A and B and its fixed-order reductions
// into dst[0] (dst[0..4] with `metrics`).
int enqueue_objective(nmd_ctx* c, hipStream_t st, bool metrics, double* dst) {
  const Side& sd = c->ws;
  const int64_t rw = nmd::dense_rows_per_wg(c->rp);
  const int64_t units = ((c->m + rw - 1) / rw) * sd.nblk();
  int64_t min_len = c->n;
  for (int32_t b = 0; b < sd.nblk(); ++b) min_len = std::min(min_len, sd.bounds[b + 1] - sd.bounds[b]);
  int nsub = (int)std::min<int64_t>(kObjSubMax, std::max<int64_t>(1, (kTargetWgs + units - 1) / units));
  nsub = (int)std::max<int64_t>(1, std::min<int64_t>(nsub, min_len / 16));
  int64_t npart = 0;
  HIP_TRY(c, nmd::launch_objective(c->A, c->m, c->B, sd.d_bounds, sd.nblk(), nsub, sd.d_rowptr,
                                   sd.d_idx, sd.d_val, c->rp, metrics, c->objpart, &npart, st));
  const int nq = metrics ? 5 : 1;
  if (nq * npart > c->objpart_count) return fail(c, NMD_EDEVICE, "internal: objective buffer");
  for (int k = 0; k < nq; ++k)
    HIP_TRY(c, nmd::launch_sum(c->objpart + (int64_t)k * npart, npart, dst + k, st));
  return NMD_OK;
}

// The sums of the objective kernel (one, or five with `metrics`), reduced on the device in a
// fixed order and copied to q[].
int objective_sums(nmd_ctx* c, const float* W, const float* H, hipStream_t st, bool metrics,
                   double* q) {
  int rc;
  if ((rc = ensure_device(c))) return rc;
  if ((rc = load_factors(c, W, H, st))) return rc;
  if ((rc = enqueue_objective(c, st, metrics, c->objout))) return rc;
  const int nq = metrics ? 5 : 1;
  HIP_TRY(c, hipMemcpyAsync(c->h_obj, c->objout, nq * sizeof(double), hipMemcpyDeviceToHost, st));
  HIP_TRY(c, hipStreamSynchronize(st));
  for (int k = 0; k < 5; ++k) q[k] = k < nq ? c->h_obj[k] : 0.0;
  return NMD_OK;
}

// Enqueues the steps of one sweep (its block list, or the two full half-steps in deterministic
// mode) with step ids from *step_id on.
int enqueue_sweep(nmd_ctx* c, const std::vector<int32_t>& list, bool full_halves, int* step_id,
                  hipStream_t st) {
  int rc;
  if (full_halves) {
    const int32_t all = -1;
    for (const bool w : {true, false}) {
      if ((rc = factor_run(c, w, &all, 1, *step_id, st))) return rc;
      if ((rc = factor_step(c, w, -1, c->opt.eta, c->opt.momentum, *step_id, c->Gneg[0], st)))
        return rc;
      *step_id += (int)(w ? c->ws.nblk() : c->hs.nblk());
    }
    return NMD_OK;
  }
  // runs of consecutive steps of one side, at most kSolveBatch long
  size_t i = 0;
  while (i < list.size()) {
    const bool w = list[i] > 0;
    int32_t blocks[nmd::kSolveBatch];
    int n = 0;
    while (i + n < list.size() && n < nmd::kSolveBatch && (list[i + n] > 0) == w) {
      blocks[n] = (w ? list[i + n] : -list[i + n]) - 1;
      ++n;
    }
    if ((rc = factor_run(c, w, blocks, n, *step_id, st))) return rc;
    for (int b = 0; b < n; ++b) {
      if ((rc = factor_step(c, w, blocks[b], c->opt.eta, c->opt.momentum, *step_id, c->Gneg[b],
                            st)))
        return rc;
      ++*step_id;
    }
    i += n;
  }
  return NMD_OK;
}

int run(nmd_ctx* c, float* W, float* H, const std::vector<std::vector<int32_t>>& lists,
        bool full_halves, hipStream_t st) {
  int rc = ensure_device(c);
  if (rc) return rc;
  if ((rc = load_factors(c, W, H, st))) return rc;
  c->enqueued.clear();
  int step_id = 0;
  for (const auto& list : lists)
    if ((rc = enqueue_sweep(c, list, full_halves, &step_id, st))) return rc;
  return NMD_OK;
}

// Sweeps with the objective evaluated on the device after each one (NMD_FLAG_SWEEP_OBJECTIVE)
// and, with `guard`, the step-size safeguard of NMD_FLAG_GUARD: before each sweep the factors
// are copied aside; after it a one-thread kernel compares the objective with the one before
// and flags a rise in the status word, which stops every later step and copy of the call.
// When the call's work has run the host reads the status once: on a rise it restores the
// factors from the copies, clears the momenta, halves eta and enqueues the remaining sweeps
// again from the rejected one (same sweep counter, same block order).
int sweeps_tracked(nmd_ctx* c, float* W, float* H, int32_t n_sweeps, hipStream_t st, bool guard) {
  int rc = ensure_device(c);
  if (rc) return rc;
  const bool sto = c->opt.mode == NMD_STOCHASTIC;
  const int32_t steps_per = c->hs.nblk() + c->ws.nblk();
  const int64_t ma = (c->m + 256) * (int64_t)c->rp, nb = (c->n + 256) * (int64_t)c->rp;
  if (c->fhist_cap < (int64_t)n_sweeps + 1) {
    dfree(c->fhist);
    c->fhist_cap = 0;
    if (dalloc(&c->fhist, (int64_t)n_sweeps + 1) != hipSuccess)
      return fail(c, NMD_ENOMEM, "device allocation of the objective history failed");
    c->fhist_cap = (int64_t)n_sweeps + 1;
  }
  if (guard && (!c->SA || !c->SB)) {
    if (dalloc(&c->SA, ma) != hipSuccess || dalloc(&c->SB, nb) != hipSuccess) {
      dfree(c->SA);
      dfree(c->SB);
      return fail(c, NMD_ENOMEM, "device allocation of the safeguard copies failed");
    }
  }
  c->fcount = 0;
  if ((rc = load_factors(c, W, H, st))) return rc;
  if ((rc = enqueue_objective(c, st, false, c->fhist))) return rc;
  const float eta_floor = c->opt.eta_min > 0.0f ? c->opt.eta_min : c->eta0 / 1024.0f;
  const double tol2 = (1.0 + (double)c->opt.guard_tol) * (1.0 + (double)c->opt.guard_tol);
  int32_t done = 0;
  while (done < n_sweeps) {
    const int64_t first = c->t;
    c->enqueued.clear();
    int step_id = 0;
    for (int32_t s = done; s < n_sweeps; ++s) {
      const std::vector<int32_t> list =
          make_schedule(c->seed, first + (s - done), c->hs.nblk(), c->ws.nblk(), sto);
      if (guard) {
        HIP_TRY(c, nmd::launch_guarded_copy(c->A, c->SA, ma, c->status, st));
        HIP_TRY(c, nmd::launch_guarded_copy(c->B, c->SB, nb, c->status, st));
      }
      const int sweep_first_step = step_id;
      if ((rc = enqueue_sweep(c, list, !sto, &step_id, st))) return rc;
      if ((rc = enqueue_objective(c, st, false, c->fhist + s + 1))) return rc;
      if (guard)
        HIP_TRY(c, nmd::launch_guard(c->fhist + s, c->fhist + s + 1, tol2, c->status,
                                     sweep_first_step, st));
    }
    if ((c->opt.flags & NMD_FLAG_ASYNC) && !guard) {
      c->t += n_sweeps - done;
      c->fcount = (int64_t)n_sweeps + 1;
      return store_factors(c, W, H, st);
    }
    HIP_TRY(c, hipMemcpyAsync(c->h_status, c->status, 2 * sizeof(int), hipMemcpyDeviceToHost, st));
    HIP_TRY(c, hipStreamSynchronize(st));
    const int flags = c->h_status[0];
    if (flags == 0) {
      c->t += n_sweeps - done;
      done = n_sweeps;
      break;
    }
    const int step = nmd::status_step(c->h_status[1]);
    const int32_t bad = done + step / steps_per;  // the sweep of the first failure
    if (nmd::status_kind(c->h_status[1]) == nmd::STATUS_RISE) {
      // every step after the rise wrote nothing: the copies hold the factors before sweep `bad`
      HIP_TRY(c, hipMemcpyAsync(c->A, c->SA, (size_t)ma * sizeof(float), hipMemcpyDeviceToDevice, st));
      HIP_TRY(c, hipMemcpyAsync(c->B, c->SB, (size_t)nb * sizeof(float), hipMemcpyDeviceToDevice, st));
      HIP_TRY(c, nmd::launch_zero(c->VA, ma, st));
      HIP_TRY(c, nmd::launch_zero(c->VB, nb, st));
      HIP_TRY(c, hipMemsetAsync(c->status, 0, sizeof(int), st));
      HIP_TRY(c, hipMemsetAsync(c->status + 1, 0x7f, sizeof(int), st));
      c->t = first + (bad - done);
      c->rejected += 1;
      const float eta_old = c->opt.eta;
      c->opt.eta = 0.5f * eta_old;
      done = bad;
      if (c->opt.eta < eta_floor) {
        c->opt.eta = eta_old;
        c->fcount = (int64_t)done + 1;
        if ((rc = store_factors(c, W, H, st))) return rc;
        HIP_TRY(c, hipStreamSynchronize(st));
        return fail(c, NMD_ESTEP,
                    "sweep %lld raised the objective at eta = %g; halving would go below %g",
                    (long long)c->t, (double)eta_old, (double)eta_floor);
      }
      continue;
    }
    // a step rejected by the device (Gram not positive definite, non-finite factor)
    c->fcount = (int64_t)bad + 1;
    rc = conclude(c, W, H, st, first, steps_per);  // step ids of this round start at `first`
    c->t = first + (bad - done);
    return rc;
  }
  c->fcount = (int64_t)n_sweeps + 1;
  if ((rc = store_factors(c, W, H, st))) return rc;
  HIP_TRY(c, hipStreamSynchronize(st));
  return NMD_OK;
}

}  // namespace

int nmd::set_static_error(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_create_error = buf;
  return code;
}

void nmd::clear_static_error() { g_create_error.clear(); }

// =================================================================================== ABI ==
extern "C" {

int nmd_create(nmd_ctx** out, int64_t m, int64_t n, int32_t r, int32_t block_m, int32_t block_n,
               uint64_t seed, const nmd_options* opts) {
  g_create_error.clear();
  if (!out) return fail(nullptr, NMD_EINVAL, "out must be non-NULL");
  *out = nullptr;
  if (m < 1 || n < 1 || m > INT32_MAX || n > INT32_MAX)
    return fail(nullptr, NMD_EINVAL, "m and n must lie in [1, 2^31-1] (got %lld, %lld)",
                (long long)m, (long long)n);
  if (r < 1 || r > 512 || r > m || r > n)
    return fail(nullptr, NMD_EINVAL, "rank r = %d must satisfy 1 <= r <= min(m, n, 512)", r);
  if (block_m < 1 || block_n < 1)
    return fail(nullptr, NMD_EINVAL, "block sizes must be >= 1");
  nmd_options o{sizeof(nmd_options), NMD_DETERMINISTIC, 1.0f, 0.0f, 0u, 0.0f, 0.0f};
  if (opts) {
    // the five-field form (through `flags`) is accepted; the later fields keep their defaults
    const uint32_t five = (uint32_t)offsetof(nmd_options, guard_tol);
    if (opts->size < five)
      return fail(nullptr, NMD_EINVAL, "opts->size = %u is smaller than %u", opts->size, five);
    std::memcpy(&o, opts, std::min<size_t>(opts->size, sizeof(nmd_options)));
    o.size = sizeof(nmd_options);
  }
  if (o.mode != NMD_DETERMINISTIC && o.mode != NMD_STOCHASTIC)
    return fail(nullptr, NMD_EINVAL, "unknown mode %d", o.mode);
  if (!(o.eta >= 0.0f) || !std::isfinite(o.eta))
    return fail(nullptr, NMD_EINVAL, "eta must be finite and >= 0");
  if (!(o.momentum >= 0.0f && o.momentum < 1.0f))
    return fail(nullptr, NMD_EINVAL, "momentum must lie in [0, 1)");
  if (o.flags & ~(uint32_t)(NMD_FLAG_ASYNC | NMD_FLAG_TIMING | NMD_FLAG_SPLIT_BF16 |
                            NMD_FLAG_SWEEP_OBJECTIVE | NMD_FLAG_GUARD))
    return fail(nullptr, NMD_EINVAL, "unknown option flags 0x%x", o.flags);
  if (!(o.guard_tol >= 0.0f) || !std::isfinite(o.guard_tol))
    return fail(nullptr, NMD_EINVAL, "guard_tol must be finite and >= 0");
  if (!(o.eta_min >= 0.0f) || !std::isfinite(o.eta_min))
    return fail(nullptr, NMD_EINVAL, "eta_min must be finite and >= 0");
  std::vector<int64_t> rb = balanced_bounds(m, block_m), cb = balanced_bounds(n, block_n);
  int64_t min_rb = m, min_cb = n;
  for (size_t k = 0; k + 1 < rb.size(); ++k) min_rb = std::min(min_rb, rb[k + 1] - rb[k]);
  for (size_t k = 0; k + 1 < cb.size(); ++k) min_cb = std::min(min_cb, cb[k + 1] - cb[k]);
  if (o.mode == NMD_STOCHASTIC && (r > min_rb || r > min_cb))
    return fail(nullptr, NMD_EINVAL,
                "rank %d exceeds the smallest block (%lld rows, %lld columns): singular Gram",
                r, (long long)min_rb, (long long)min_cb);
  nmd_ctx* c = new (std::nothrow) nmd_ctx();
  if (!c) return fail(nullptr, NMD_ENOMEM, "context allocation failed");
  c->m = m;
  c->n = n;
  c->r = r;
  c->rp = nmd::padded_rank(r);
  c->block_m = block_m;
  c->block_n = block_n;
  c->seed = seed;
  c->opt = o;
  c->eta0 = o.eta;
  c->rb = std::move(rb);
  c->cb = std::move(cb);
  *out = c;
  return NMD_OK;
}

int nmd_set_sparse_csr(nmd_ctx* c, int64_t nnz, const int64_t* row_ptr, const int32_t* col_idx,
                       const float* values) {
  if (!c) return NMD_EINVAL;
  c->err.clear();
  if (nnz < 0) return fail(c, NMD_EINVAL, "nnz must be >= 0");
  if (!row_ptr) return fail(c, NMD_EINVAL, "row_ptr must be non-NULL");
  if (nnz > 0 && (!col_idx || !values))
    return fail(c, NMD_EINVAL, "col_idx and values must be non-NULL when nnz > 0");
  if (nnz >= INT32_MAX) return fail(c, NMD_EINVAL, "nnz must be < 2^31-1");
  const int64_t m = c->m, n = c->n;
  nmd::Compressed rows, cols;
  double s2 = 0.0;
  try {
    const std::string why = nmd::ingest_csr(m, n, nnz, row_ptr, col_idx, values, rows, cols, &s2);
    if (!why.empty()) return fail(c, NMD_EINVAL, "%s", why.c_str());
  } catch (const std::bad_alloc&) {
    return fail(c, NMD_ENOMEM, "host allocation failed while arranging S");
  }
  const int64_t nz = (int64_t)rows.idx.size();
  free_sparse_device(c);
  c->has_S = false;
  try {
    nmd::build_side(c->ws, m, n, c->cb, rows.ptr.data(), rows.idx.data(), rows.val.data());
    nmd::build_side(c->hs, n, m, c->rb, cols.ptr.data(), cols.idx.data(), cols.val.data());
  } catch (const std::bad_alloc&) {
    return fail(c, NMD_ENOMEM, "host allocation failed while arranging S");
  }
  c->nnz_col_blocks.assign(c->ws.nblk(), 0);
  c->nnz_row_blocks.assign(c->hs.nblk(), 0);
  for (int32_t b = 0; b < c->ws.nblk(); ++b)
    c->nnz_col_blocks[b] = c->ws.entry_off[b + 1] - c->ws.entry_off[b];
  for (int32_t b = 0; b < c->hs.nblk(); ++b)
    c->nnz_row_blocks[b] = c->hs.entry_off[b + 1] - c->hs.entry_off[b];
  c->nnz = nz;
  c->s_norm = std::sqrt(s2);
  c->has_S = true;
  return NMD_OK;
}

int nmd_als_block_sweep(nmd_ctx* c, float* W, float* H, int32_t n_sweeps, void* hip_stream) {
  int rc = check_ready(c, W, H);
  if (rc) return rc;
  if (n_sweeps < 1) return fail(c, NMD_EINVAL, "n_sweeps must be >= 1");
  hipStream_t st = (hipStream_t)hip_stream;
  const bool sto = c->opt.mode == NMD_STOCHASTIC;
  const int32_t steps_per = c->hs.nblk() + c->ws.nblk();
  if ((int64_t)n_sweeps * steps_per > kMaxStepsPerCall)
    return fail(c, NMD_EINVAL, "%d sweeps of %d steps exceed %lld steps per call; split the call",
                n_sweeps, steps_per, (long long)kMaxStepsPerCall);
  const bool guard = (c->opt.flags & NMD_FLAG_GUARD) != 0;
  if (!guard && !(c->opt.flags & NMD_FLAG_SWEEP_OBJECTIVE)) {
    std::vector<std::vector<int32_t>> lists;
    for (int32_t s = 0; s < n_sweeps; ++s)
      lists.push_back(make_schedule(c->seed, c->t + s, c->hs.nblk(), c->ws.nblk(), sto));
    const int64_t first = c->t;
    rc = run(c, W, H, lists, !sto, st);
    if (rc) return rc;
    c->t += n_sweeps;
    rc = conclude(c, W, H, st, first, steps_per);
    if (rc == NMD_ENOTPD || rc == NMD_ENONFINITE) c->t = first + c->last_fail_step / steps_per;
    return rc;
  }
  return sweeps_tracked(c, W, H, n_sweeps, st, guard);
}

int nmd_run_steps(nmd_ctx* c, float* W, float* H, const int32_t* steps, int32_t n_steps,
                  void* hip_stream) {
  int rc = check_ready(c, W, H);
  if (rc) return rc;
  if (n_steps < 0 || (n_steps > 0 && !steps)) return fail(c, NMD_EINVAL, "bad step list");
  if (n_steps > kMaxStepsPerCall)
    return fail(c, NMD_EINVAL, "%d steps exceed %lld steps per call; split the call", n_steps,
                (long long)kMaxStepsPerCall);
  for (int32_t k = 0; k < n_steps; ++k) {
    const int32_t code = steps[k];
    if (code == 0 || (code > 0 && code > c->ws.nblk()) || (code < 0 && -code > c->hs.nblk()))
      return fail(c, NMD_EINVAL, "step code %d out of range", code);
  }
  std::vector<std::vector<int32_t>> lists(1, std::vector<int32_t>(steps, steps + n_steps));
  rc = run(c, W, H, lists, false, (hipStream_t)hip_stream);
  if (rc) return rc;
  return conclude(c, W, H, (hipStream_t)hip_stream, 0, 0);
}

int nmd_objective(nmd_ctx* c, const float* W, const float* H, double* out_obj, void* hip_stream) {
  int rc = check_ready(c, W, H);
  if (rc) return rc;
  if (!out_obj) return fail(c, NMD_EINVAL, "out_obj must be non-NULL");
  double q[5];
  if ((rc = objective_sums(c, W, H, (hipStream_t)hip_stream, false, q))) return rc;
  *out_obj = std::sqrt(std::max(q[0], 0.0)) / c->s_norm;
  return NMD_OK;
}

int nmd_metrics(nmd_ctx* c, const float* W, const float* H, double* out, void* hip_stream) {
  int rc = check_ready(c, W, H);
  if (rc) return rc;
  if (!out) return fail(c, NMD_EINVAL, "out must be non-NULL");
  double q[5];
  if ((rc = objective_sums(c, W, H, (hipStream_t)hip_stream, true, q))) return rc;
  const double s2 = c->s_norm;
  out[0] = std::sqrt(std::max(q[0] + q[1], 0.0)) / s2;
  out[1] = std::sqrt(std::max(q[0] + q[2], 0.0)) / s2;
  out[2] = q[4] > 0.0 ? 1.0 - q[3] / q[4] : 1.0;
  return NMD_OK;
}

void nmd_destroy(nmd_ctx* c) {
  if (!c) return;
  if (c->dev_ready) (void)hipSetDevice(c->device);
  free_device(c);
  delete c;
}

const char* nmd_last_error(const nmd_ctx* c) {
  return c ? c->err.c_str() : g_create_error.c_str();
}

int nmd_get_schedule(const nmd_ctx* c, int64_t sweep, int32_t* out, int64_t cap) {
  if (!c || !out || sweep < 0) return NMD_EINVAL;
  const int32_t R = (int32_t)c->rb.size() - 1, C = (int32_t)c->cb.size() - 1;
  if (cap < (int64_t)R + C) return NMD_EINVAL;
  const std::vector<int32_t> s = make_schedule(c->seed, sweep, R, C, c->opt.mode == NMD_STOCHASTIC);
  std::copy(s.begin(), s.end(), out);
  return (int)s.size();
}

int nmd_get_block_nnz(const nmd_ctx* c, int32_t side, int64_t* out, int64_t cap) {
  if (!c || !out || (side != 0 && side != 1)) return NMD_EINVAL;
  if (!c->has_S) return NMD_ESTATE;
  const std::vector<int64_t>& v = side == 0 ? c->nnz_col_blocks : c->nnz_row_blocks;
  if (cap < (int64_t)v.size()) return NMD_EINVAL;
  std::copy(v.begin(), v.end(), out);
  return (int)v.size();
}

int nmd_get_block_bounds(const nmd_ctx* c, int32_t side, int64_t* out, int64_t cap) {
  if (!c || !out || (side != 0 && side != 1)) return NMD_EINVAL;
  const std::vector<int64_t>& v = side == 0 ? c->cb : c->rb;
  if (cap < (int64_t)v.size()) return NMD_EINVAL;
  std::copy(v.begin(), v.end(), out);
  return (int)v.size();
}

int nmd_reset(nmd_ctx* c) {
  if (!c) return NMD_EINVAL;
  c->err.clear();
  c->t = 0;
  c->opt.eta = c->eta0;
  c->rejected = 0;
  c->fcount = 0;
  if (c->dev_ready) {
    HIP_TRY(c, hipSetDevice(c->device));
    HIP_TRY(c, hipDeviceSynchronize());
    HIP_TRY(c, hipMemset(c->VA, 0, (size_t)(c->m + 256) * c->rp * sizeof(float)));
    HIP_TRY(c, hipMemset(c->VB, 0, (size_t)(c->n + 256) * c->rp * sizeof(float)));
    HIP_TRY(c, hipMemset(c->status, 0, sizeof(int)));
    HIP_TRY(c, hipMemset(c->status + 1, 0x7f, sizeof(int)));
    HIP_TRY(c, hipDeviceSynchronize());
  }
  return NMD_OK;
}

int nmd_get_sweep_objectives(nmd_ctx* c, double* out, int64_t cap) {
  if (!c || (!out && cap > 0)) return NMD_EINVAL;
  c->err.clear();
  if (c->fcount == 0) return 0;
  if (cap < c->fcount) return fail(c, NMD_EINVAL, "cap %lld < %lld objectives", (long long)cap,
                                   (long long)c->fcount);
  HIP_TRY(c, hipSetDevice(c->device));
  HIP_TRY(c, hipDeviceSynchronize());
  HIP_TRY(c, hipMemcpy(out, c->fhist, (size_t)c->fcount * sizeof(double), hipMemcpyDeviceToHost));
  for (int64_t k = 0; k < c->fcount; ++k) out[k] = std::sqrt(std::max(out[k], 0.0)) / c->s_norm;
  return (int)c->fcount;
}

int nmd_get_step_size(const nmd_ctx* c, float* eta, int64_t* rejected) {
  if (!c || !eta) return NMD_EINVAL;
  *eta = c->opt.eta;
  if (rejected) *rejected = c->rejected;
  return NMD_OK;
}

int nmd_get_sweep_count(const nmd_ctx* c, int64_t* t) {
  if (!c || !t) return NMD_EINVAL;
  *t = c->t;
  return NMD_OK;
}

int nmd_rectified_contraction(const float* A, int64_t rows, const float* B, int64_t blk,
                              int32_t r, float* Y, void* hip_stream) {
  g_create_error.clear();
  if (!A || !B || !Y) return fail(nullptr, NMD_EINVAL, "A, B and Y must be non-NULL");
  if (rows < 1 || blk < 1 || rows > INT32_MAX)
    return fail(nullptr, NMD_EINVAL, "rows and blk must be >= 1");
  if (r < 16 || r > 512 || nmd::padded_rank(r) != r)
    return fail(nullptr, NMD_EINVAL,
                "r = %d unsupported: use 16, 32, 48, 64 or a multiple of 64 up to 512", r);
  hipError_t e =
      nmd::launch_dense(A, rows, B, blk, r, Y, 0, 1, 1.0f, nullptr, (hipStream_t)hip_stream);
  if (e != hipSuccess) return fail(nullptr, NMD_EDEVICE, "launch failed: %s", hipGetErrorString(e));
  return NMD_OK;
}

int64_t nmd_bf16x3_workspace_floats(int64_t blk, int32_t r) {
  if (blk < 1 || !nmd::bf16x3_rank(r)) return -1;
  return nmd::bf16x3_work_floats(blk, r);
}

int nmd_rectified_contraction_bf16x3(const float* A, int64_t rows, const float* B, int64_t blk,
                                     int32_t r, float* work, float* Y, void* hip_stream) {
  g_create_error.clear();
  if (!A || !B || !work || !Y)
    return fail(nullptr, NMD_EINVAL, "A, B, work and Y must be non-NULL");
  if (rows < 1 || blk < 1 || rows > INT32_MAX)
    return fail(nullptr, NMD_EINVAL, "rows and blk must be >= 1");
  if (!nmd::bf16x3_rank(r))
    return fail(nullptr, NMD_EINVAL,
                "the bf16x3 contraction needs r in {16, 32, 64, 128, 256, 512} (got %d)", r);
  hipError_t e = nmd::launch_bf16x3(A, rows, B, blk, r, work, Y, 0, 1, 1.0f, nullptr,
                                    (hipStream_t)hip_stream);
  if (e != hipSuccess) return fail(nullptr, NMD_EDEVICE, "launch failed: %s", hipGetErrorString(e));
  return NMD_OK;
}

int nmd_get_kernel_timing(nmd_ctx* c, int32_t kernel, double* total_ms, int64_t* launches,
                          double* flops, double* bytes, int32_t reset) {
  if (!c || kernel < 0 || kernel >= K_COUNT) return NMD_EINVAL;
  int rc = collect_timing(c);
  if (rc) return rc;
  if (total_ms) *total_ms = c->t_ms[kernel];
  if (launches) *launches = c->t_launch[kernel];
  if (flops) *flops = c->t_flops[kernel];
  if (bytes) *bytes = c->t_bytes[kernel];
  if (reset) {
    for (int k = 0; k < K_COUNT; ++k) {
      c->t_ms[k] = 0;
      c->t_launch[k] = 0;
      c->t_flops[k] = 0;
      c->t_bytes[k] = 0;
    }
  }
  return NMD_OK;
}

int nmd_get_dense_blocks(nmd_ctx* c, int64_t* run, int64_t* total, int64_t* entries,
                         int32_t reset) {
  if (!c) return NMD_EINVAL;
  unsigned long long v[2] = {0, 0};
  if (c->dev_ready) {
    HIP_TRY(c, hipSetDevice(c->device));
    HIP_TRY(c, hipDeviceSynchronize());
    HIP_TRY(c, hipMemcpy(v, c->g2, sizeof v, hipMemcpyDeviceToHost));
  }
  if (run) *run = (int64_t)v[0];
  if (total) *total = c->g2_total;
  if (entries) *entries = (int64_t)v[1];
  if (reset) {
    if (c->dev_ready) {
      HIP_TRY(c, hipMemset(c->g2, 0, sizeof v));
      HIP_TRY(c, hipDeviceSynchronize());
    }
    c->g2_total = 0;
  }
  return NMD_OK;
}

}  // extern "C"
