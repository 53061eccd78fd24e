// Internal declarations shared by the host driver and the HIP kernels of libnmd.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ingest.h"

namespace nmd {

// Device status word: status[0] is the union of the flag bits raised; status[1] the smallest
// step_id * 8 + bit among them, so it names the first failing step and why it failed.  A
// failure stops the step that raised it and every step after it (step_blocked), but not the
// steps before it, whose work may be enqueued behind the check that failed (the solves of a run
// of steps are formed ahead of their applies).
enum { STATUS_NOTPD = 1, STATUS_NONFINITE = 2, STATUS_RISE = 4 };
inline int status_step(int word) { return word >> 3; }
inline int status_kind(int word) { return word & 7; }
__device__ __forceinline__ void flag_status(int* status, int bit, int step_id) {
  atomicOr(&status[0], bit);
  atomicMin(&status[1], step_id * 8 + bit);
}
__device__ __forceinline__ bool step_blocked(const int* status, int step_id) {
  return *(volatile const int*)status != 0 &&
         (*(volatile const int*)(status + 1) >> 3) <= step_id;
}

// The solves of up to kSolveBatch consecutive steps of one side, formed in one set of
// launches: matrix b is the Gram matrix of panel rows j0[b] .. j0[b] + blk[b] of step
// step_id[b].
constexpr int kSolveBatch = 8;
struct SolveBatch {
  int n;
  int step_id[kSolveBatch];
  int64_t j0[kSolveBatch];
  int64_t blk[kSolveBatch];
};

// Padded rank: the kernels work on r_p columns (zeros beyond r).
int padded_rank(int r);
// Rows per workgroup of the dense kernel for padded rank rp.
int dense_rows_per_wg(int rp);

// Workgroups of the dense kernel for padded rank rp that one CU holds at once.
hipError_t dense_wgs_per_cu(int rp, int* out);
// The same two for r_p >= 320, whose instantiations are in their own translation unit.
hipError_t dense_wgs_per_cu_large(int rp, int* out);
hipError_t launch_dense_large(const float* X, int64_t rows, const float* P, int64_t blk, int rp,
                              float* Ypart, int64_t y_stride, int nsplit, float sgn,
                              unsigned long long* gemm2_blocks, hipStream_t st);

// Y_s = sgn * max(0, X P^T) P over the split s of the rows of P (rows of X: `rows`).  Ypart
// holds nsplit buffers of y_stride floats each (row-major rows x rp).  When gemm2_blocks is not
// NULL it receives (atomically) the number of slices (16 rows x 4 panel rows) that ran the
// second contraction; the others had no positive L entry and were skipped.
hipError_t launch_dense(const float* X, int64_t rows, const float* P, int64_t blk, int rp,
                        float* Ypart, int64_t y_stride, int nsplit, float sgn,
                        unsigned long long* gemm2_blocks, hipStream_t st);

// Both products on split bf16 MFMA (dense_bf16.h), rp in {16, 32, 64, 128, 256, 512}
// (bf16x3_rank): splits the blk x rp
// panel P into `work` (bf16x3_work_floats(blk, rp) floats: row-major and transposed split
// copies), then Y_s = sgn * max(0, X P_s^T) P_s for each of nsplit panel ranges starting at
// bf16x3_pair_start(s, nsplit, blk) (whole 32-row pairs).  When `live` is not NULL, 8 per
// 16 x 32 tile of max(0, L) with a positive entry is added to it (its 16 x 4 slices).
bool bf16x3_rank(int rp);
int64_t bf16x3_work_floats(int64_t blk, int rp);
int64_t bf16x3_pair_start(int s, int nsplit, int64_t blk);
hipError_t launch_bf16x3(const float* X, int64_t rows, const float* P, int64_t blk, int rp,
                         float* work, float* Ypart, int64_t y_stride, int nsplit, float sgn,
                         unsigned long long* live, hipStream_t st);
// The rp = 256 and 512 form (dense_bf16_large.hip), same contract; at these ranks `work` holds
// only the row-major split copy (bf16x3_work_floats = blk * rp).
hipError_t launch_bf16x3_staged(const float* X, int64_t rows, const float* P, int64_t blk, int rp,
                                float* work, float* Ypart, int64_t y_stride, int nsplit,
                                float sgn, unsigned long long* live, hipStream_t st);

// Sparse correction: for every item, c = sum over its entries of (s - min(0, x_row . p_j)) p_j;
// a row with a single item gets Y[row] = c (accumulate = 0) or Y[row] += c (accumulate = 1);
// a row split over several items has its slots summed in order by the fix-up, which writes or
// adds the same way.
hipError_t launch_sparse(const Item* items, int64_t nitems, const int32_t* idx, const float* val,
                         const float* X, const float* P, int rp, float* Y, float* scratch,
                         int accumulate, hipStream_t st);
hipError_t launch_fixup(const Split* splits, int64_t nsplits, const float* scratch, int rp,
                        float* Y, int accumulate, hipStream_t st);

// Gram matrices G_b = P_b^T P_b (fp64, rp x rp, identity on the padded diagonal) of the panel
// row ranges of a batch, G_b at G + b rp^2; Gpart holds sb.n * nchunks * rp^2 doubles.
hipError_t launch_gram(const float* P, const SolveBatch& sb, int r, int rp, double* Gpart,
                       int nchunks, double* G, hipStream_t st);
// -G_b^-1 through the Cholesky factorisation G_b = L L^T (chol.hip) for each matrix of a batch
// (G_b at G + b rp^2): result[b] receives -G_b^-1 (rp x rp, inside `work`, which holds
// sb.n * chol_work_doubles(rp) doubles); a non-positive pivot flags status with the step id of
// its matrix.
int64_t chol_work_doubles(int rp);
hipError_t launch_chol_inverse(const double* G, double* work, int rp, int* status,
                               const SolveBatch& sb, double** result, hipStream_t st);
// The same with one workgroup per matrix doing all three steps in one launch.
hipError_t launch_chol_inverse_fused(const double* G, double* work, int rp, int* status,
                                     const SolveBatch& sb, double** result, hipStream_t st);
// Vout = gamma Vin + eta U (-Gneg), Xout = Xin + Vout, where U = Delta P_J is the sum (fp64)
// of the nsplit partial outputs plus, when Ysp is not NULL, a separate correction buffer
// (rows x rp), and -Gneg = (P_J^T P_J)^-1.  The outputs are other buffers than the inputs, so
// a step that a later check rejects leaves its inputs intact.  Nothing is written once status
// holds a failure of this step or an earlier one.
hipError_t launch_apply(const float* Ypart, int64_t y_stride, int nsplit, const float* Ysp,
                        const double* Gneg, const float* Xin, const float* Vin, float* Xout,
                        float* Vout, int64_t rows, int rp, float eta, float gamma, int* status,
                        int step_id, hipStream_t st);

// Layout helpers between the caller's W (m x r), H (r x n) and the padded panels.
hipError_t launch_pad_rows(const float* src, int64_t rows, int r, float* dst, int rp,
                           hipStream_t st);
hipError_t launch_unpad_rows(const float* src, int64_t rows, int rp, float* dst, int r,
                             hipStream_t st);
hipError_t launch_transpose_in(const float* H, int r, int64_t n, float* B, int rp,
                               hipStream_t st);
hipError_t launch_transpose_out(const float* B, int rp, int64_t n, float* H, int r,
                                hipStream_t st);
hipError_t launch_zero(float* p, int64_t count, hipStream_t st);
// dst = src (count floats) unless status[0] is already set.
hipError_t launch_guarded_copy(const float* src, float* dst, int64_t count, const int* status,
                               hipStream_t st);
// Step-size safeguard: unless status[0] is already set, flags STATUS_RISE with step_id when
// *q_new is not <= tol2 * *q_old (objective sums of squares; NaN counts as a rise).
hipError_t launch_guard(const double* q_old, const double* q_new, double tol2, int* status,
                        int step_id, hipStream_t st);

// Objective: per-workgroup fp64 sums of the eq. SLloss terms over (row tile, column block,
// sub-split); rowptr holds, per column block, the row pointers of the W-side entries.  With
// `metrics`, five sums (objective and reconstruction measures) laid out as
// partial[k * npartial + workgroup], k = 0..4; otherwise one.
hipError_t launch_objective(const float* X, int64_t rows, const float* P, const int64_t* cbounds,
                            int nblk, int nsub, const int64_t* rowptr, const int32_t* idx,
                            const float* val, int rp, bool metrics, double* partial,
                            int64_t* npartial, hipStream_t st);
hipError_t launch_sum(const double* partial, int64_t count, double* out, hipStream_t st);

int dense_max_wgs(int64_t rows, int rp, int nsplit);

// The message nmd_last_error(NULL) returns for the entry points without a context: sets it and
// returns `code`, or clears it.
int set_static_error(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_static_error();

}  // namespace nmd
