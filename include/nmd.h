/*
 * nmd.h - C ABI of an MI355X (gfx950) library for stochastic alternating least squares (SALSA)
 * in subzero matrix completion: given a sparse nonnegative S (m x n), fit real factors W (m x r)
 * and H (r x n) so that S ~ max(0, W H).
 *
 * The method (Saul et al., "Subzero matrix completion for sparse data analysis"):
 *   L = W H (eq. ABt, with A = W and B = H^T), S-hat = max(0, L) (eq. rectify),
 *   Z = S on the nonzeros of S and L - S-hat = min(0, L) elsewhere (eq. updateZ),
 *   least-squares factor updates A <- Z B (B^T B)^-1, B <- Z^T A (A^T A)^-1 (eqs. lsqA, lsqB),
 *   their stochastic form on a column mini-batch J, A <- A + eta Delta_{:J} B_J [B_J^T B_J]^-1
 *   (eqs. Shat_sto, Delta_sto, lsqA_sto), the analogous update of B on a row mini-batch I, and a
 *   heavy-ball momentum term, gamma times the last step taken (Sec. 4.1).
 *   Objective: ||Z - L||_F / ||S||_F (eq. auxCost) with Z eliminated as in eq. SLloss.
 *
 * Every entry point returns an int status (NMD_OK or a negative code); no C++ exception
 * crosses this boundary.  Argument errors are detected before any device work is enqueued, so
 * caller buffers are left untouched.  A context is not thread-safe; distinct contexts are
 * independent.  All device pointers must be allocated on the device that is current when the
 * context first touches the GPU (the device is remembered and made current on each call).
 */
#ifndef NMD_H
#define NMD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct nmd_ctx nmd_ctx; /* opaque */

enum {
  NMD_OK = 0,
  NMD_EINVAL = -1,     /* bad argument (sizes, pointers, CSR structure, values)            */
  NMD_ENOMEM = -2,     /* host or device allocation failed                                 */
  NMD_EDEVICE = -3,    /* a HIP runtime call failed or no usable gfx950 device             */
  NMD_ENOTPD = -4,     /* a Gram matrix B_J^T B_J or A_I^T A_I was not positive definite    */
  NMD_ESTATE = -5,     /* call out of order (e.g. a sweep before nmd_set_sparse_csr)         */
  NMD_ENONFINITE = -6, /* an updated factor entry was NaN or infinite                      */
  NMD_ESTEP = -7       /* the step-size safeguard (NMD_FLAG_GUARD) would lower the step size
                          below eta_min                                                     */
};

enum { NMD_DETERMINISTIC = 0, NMD_STOCHASTIC = 1 };

enum {
  NMD_FLAG_ASYNC = 1u, /* do not synchronise at the end of a call that runs steps; a step
                          the device rejects is then not reported, the factors written
                          back are unspecified and later steps are skipped until
                          nmd_reset                                                       */
  NMD_FLAG_TIMING = 2u, /* record HIP events around every kernel class (see
                          nmd_get_kernel_timing); adds a few microseconds per step        */
  NMD_FLAG_SPLIT_BF16 = 4u, /* padded rank r_p in {16, 32, 64, 128, 256, 512}, i.e. r <= 32
                          or r in 49..64, 65..128, 193..256, 449..512 (other ranks ignore
                          it): both
                          products of the dense contraction,
                          L = A B_J^T and max(0, L) B_J, run on bf16 MFMA with every
                          operand split in two (x = bf16(x) + bf16(x - bf16(x)), three
                          products each, fp32 accumulation; relative error about 2^-16 of
                          the sum of the magnitudes of the terms) instead of fp32 MFMA, the
                          counterpart of the paper's TF32 kernels (Sec. 4.2); the kernel of
                          nmd_rectified_contraction_bf16x3.  Everything else stays fp32.
                          Needs nmd_bf16x3_workspace_floats(max(m, n), r_p) floats more
                          device memory.  It adds one small kernel per step, so on steps
                          too small to fill the GPU it can cost more than it saves         */
  NMD_FLAG_SWEEP_OBJECTIVE = 8u, /* evaluate the objective (as nmd_objective) on the device
                          before the first sweep of a call and after each sweep, into a
                          device buffer read by nmd_get_sweep_objectives; no extra
                          synchronisation.  Costs one objective evaluation per sweep         */
  NMD_FLAG_GUARD = 16u /* step-size safeguard; implies NMD_FLAG_SWEEP_OBJECTIVE.  The paper
                          notes that too large a step size makes the stochastic updates
                          diverge (Sec. 7) and lowers the step size for the models that need
                          it (appendix on experimental settings), without an automatic rule.
                          Rule used here: a sweep that leaves the objective above
                          (1 + guard_tol) times its value before the sweep, or not finite, is
                          undone (W, H and the sweep counter return to their values before
                          it), both momentum buffers are cleared, eta is halved and the sweep
                          is run again with the same block order.  Decided on the device
                          after each sweep; the host only learns of it when the call ends,
                          so the sweeps enqueued after a rejected one are skipped and
                          enqueued again.  The lowered eta persists in the context
                          (nmd_get_step_size; nmd_reset restores the initial one)            */
};

typedef struct {
  uint32_t size;     /* sizeof(nmd_options), for forward compatibility                     */
  int32_t mode;      /* NMD_DETERMINISTIC (full-batch least squares, eqs. lsqA/lsqB) or
                        NMD_STOCHASTIC (mini-batch updates, eq. lsqA_sto)                 */
  float eta;         /* step size eta > 0 of eq. lsqA_sto (1 = exact mini-batch solve)      */
  float momentum;    /* gamma in [0, 1): V <- gamma V + eta (X - A), A <- A + V            */
  uint32_t flags;    /* NMD_FLAG_* bits                                                     */
  float guard_tol;   /* NMD_FLAG_GUARD: relative rise of the objective a sweep may cause
                        before it is undone, >= 0 (0: any rise)                             */
  float eta_min;     /* NMD_FLAG_GUARD: halving that would take eta below this fails with
                        NMD_ESTEP; 0 means eta / 1024 (ten halvings)                        */
} nmd_options;
/* Defaults when opts == NULL: NMD_DETERMINISTIC, eta = 1, momentum = 0, flags = 0,
 * guard_tol = 0, eta_min = 0.  A caller built against the earlier five-field struct (size 20)
 * is accepted; the two later fields then take their defaults. */

/*
 * nmd_create - a context for an m x n problem fitted at rank r.
 *   block_m, block_n: requested row- and column-block sizes.  The rows are split into
 *     R = ceil(m / block_m) balanced blocks [floor(k m / R), floor((k+1) m / R)), the columns
 *     likewise into C blocks (the paper's row sets I and column mini-batches J, Sec. 4.1).
 *   seed: seed of the per-sweep block order (stochastic mode).
 * Requires m, n >= 1; 1 <= r <= min(m, n) and r <= 512; block sizes >= 1; in stochastic mode
 * r must not exceed the smallest row or column block (else a mini-batch Gram matrix is
 * singular).  Returns NMD_EINVAL otherwise, NMD_ENOMEM if the context cannot be allocated.
 * *out receives the context (NULL on failure).  No device memory is touched here.
 */
int nmd_create(nmd_ctx** out, int64_t m, int64_t n, int32_t r, int32_t block_m, int32_t block_n,
               uint64_t seed, const nmd_options* opts);

/*
 * nmd_set_sparse_csr - copies S (host CSR arrays; the caller may free them afterwards).
 *   row_ptr: int64[m+1], row_ptr[0] = 0, non-decreasing, row_ptr[m] = nnz.
 *   col_idx: int32[nnz], 0 <= col < n, strictly increasing within each row.
 *   values:  float[nnz], finite and >= 0.  Explicit zeros are dropped: the mask of eq. updateZ
 *            is S_ij > 0.  At least one positive value is required (||S||_F normalises the
 *            objective, eq. auxCost).
 * Builds the per-column-block rows and per-row-block columns used by the updates.  Replaces
 * any earlier S.  Returns NMD_EINVAL on a malformed matrix (S is then left unset).
 */
int nmd_set_sparse_csr(nmd_ctx* ctx, int64_t nnz, const int64_t* row_ptr, const int32_t* col_idx,
                       const float* values);

/*
 * nmd_als_block_sweep - runs n_sweeps >= 1 sweeps (epochs) in place on W and H.
 *   W: device float[m*r], row-major m x r.  H: device float[r*n], row-major r x n.
 *   hip_stream: a hipStream_t (NULL = the null stream); all work is ordered on it (the
 *   library's own streams, for the Gram matrices and inverses and, at r_p >= 320, the sparse
 *   correction, start from events on it and rejoin it before each update).
 * Stochastic mode: sweep t executes the seeded interleaved list of W-steps (one column block
 * J each, eq. lsqA_sto) and H-steps (one row block I each); see nmd_get_schedule.
 * Deterministic mode: the exact half-steps A <- A + Delta B (B^T B)^-1 over all columns, then
 * B <- B + Delta^T A (A^T A)^-1 over all rows (eqs. spLsqA, spLsqB), with eta and gamma
 * applied as in the stochastic update.  The sweep counter t and the momentum buffers persist
 * across calls (nmd_reset clears them).  Returns NMD_ESTATE without S, NMD_EINVAL on NULL
 * pointers, n_sweeps < 1 or more than 2^27 steps in the call (n_sweeps times the blocks of both
 * sides), NMD_ENOTPD / NMD_ENONFINITE when the device rejects a step: the
 * later steps are skipped, W and H receive the factors after the last completed step (the
 * momenta are kept at that state too) and nmd_last_error names the sweep and step; the sweep
 * counter then counts only the sweeps that completed.  With NMD_FLAG_GUARD, NMD_ESTEP when the
 * safeguard would lower eta below eta_min: W and H then hold the factors before the rejected
 * sweep.  NMD_EDEVICE on a HIP failure.  Unless NMD_FLAG_ASYNC is set the call synchronises the
 * stream before returning (NMD_FLAG_GUARD ignores NMD_FLAG_ASYNC: it must read the device's
 * decision).
 */
int nmd_als_block_sweep(nmd_ctx* ctx, float* W, float* H, int32_t n_sweeps, void* hip_stream);

/*
 * nmd_objective - *out_obj = sqrt(sum_{S_ij = 0} max(0, L_ij)^2 + sum_{S_ij > 0} (S_ij - L_ij)^2)
 * / ||S||_F with L = W H (eq. auxCost with Z eliminated, eq. SLloss).  W, H as in
 * nmd_als_block_sweep (read only).  Products are formed in fp32 and summed in fp64.
 * Synchronises the stream.  Errors as for nmd_als_block_sweep.
 */
int nmd_objective(nmd_ctx* ctx, const float* W, const float* H, double* out_obj, void* hip_stream);

/*
 * nmd_metrics - the objective together with the two reconstruction measures of S-hat =
 * max(0, W H) (eq. rectify), from one pass over L: out[0] = the objective of nmd_objective,
 * out[1] = ||S - S-hat||_F / ||S||_F (eq. RMSE), out[2] = 1 - sum min(S, S-hat) /
 * sum max(S, S-hat) (eq. WJD; 1 when both sums vanish).  `out` is host memory for 3 doubles.
 * W, H as in nmd_als_block_sweep (read only).  Products are formed in fp32 and summed in fp64.
 * Synchronises the stream.  Errors as for nmd_objective.
 */
int nmd_metrics(nmd_ctx* ctx, const float* W, const float* H, double* out, void* hip_stream);

/*
 * nmd_get_sweep_objectives - with NMD_FLAG_SWEEP_OBJECTIVE or NMD_FLAG_GUARD, the objectives
 * of the last nmd_als_block_sweep call: out[0] before its first sweep, out[k] after its k-th
 * (accepted) sweep, k = 1 .. n_sweeps (eq. auxCost, as nmd_objective).  `out`: host memory for
 * cap doubles.  Returns the count (n_sweeps + 1; 0 before any such call), NMD_EINVAL if cap is
 * too small.  Synchronises the device.
 */
int nmd_get_sweep_objectives(nmd_ctx* ctx, double* out, int64_t cap);

/*
 * nmd_get_step_size - the step size eta now in force (lowered by NMD_FLAG_GUARD) and, when
 * `rejected` is not NULL, the number of sweeps the safeguard has undone since nmd_create or
 * nmd_reset.
 */
int nmd_get_step_size(const nmd_ctx* ctx, float* eta, int64_t* rejected);

/* nmd_destroy - frees the context and its device memory; NULL-safe. */
void nmd_destroy(nmd_ctx* ctx);

/* ---------------------------------------------------------------- diagnostics ------------ */

/* Last error message of the context ("" if none); valid until the next call on it.  With a
 * NULL context, the message of the last failed nmd_create on this thread. */
const char* nmd_last_error(const nmd_ctx* ctx);

/*
 * nmd_get_schedule - writes the step list of sweep `sweep` (0-based) into out[0..cap) and
 * returns its length (R + C), or a negative code.  Encoding: +(k+1) is the W-step of column
 * block k, -(k+1) the H-step of row block k.  Stochastic order: SplitMix64 stream seeded with
 * seed XOR (sweep * 0x9E3779B97F4A7C15 mod 2^64), Lemire bounded integers, Fisher-Yates
 * shuffles of the C column blocks then the R row blocks, merged so that a W-step comes next
 * whenever (2w+1) R <= (2h+1) C (w, h = steps emitted so far).  Deterministic mode lists
 * +1..+C then -1..-R (the W half accumulates over every column block before one solve).
 * Host only; cap < R + C returns NMD_EINVAL.
 */
int nmd_get_schedule(const nmd_ctx* ctx, int64_t sweep, int32_t* out, int64_t cap);

/* nmd_get_block_nnz - positive entries per column block (side 0, C values) or per row block
 * (side 1, R values) into out[0..cap); returns the count or a negative code.  Host only. */
int nmd_get_block_nnz(const nmd_ctx* ctx, int32_t side, int64_t* out, int64_t cap);

/* nmd_get_block_bounds - the K+1 block offsets of the rows (side 1) or columns (side 0);
 * returns K + 1 or a negative code.  Host only. */
int nmd_get_block_bounds(const nmd_ctx* ctx, int32_t side, int64_t* out, int64_t cap);

/* nmd_reset - zeroes the momentum buffers and the sweep counter, restores the step size given
 * at creation (and the count of rejected sweeps, NMD_FLAG_GUARD), and clears a step rejection
 * left pending on the device (see NMD_FLAG_ASYNC).  Synchronises the device. */
int nmd_reset(nmd_ctx* ctx);

/* nmd_get_sweep_count - *t = number of sweeps run since creation or the last reset. */
int nmd_get_sweep_count(const nmd_ctx* ctx, int64_t* t);

/*
 * nmd_run_steps - runs the encoded steps steps[0..n_steps) (encoding of nmd_get_schedule)
 * in order, each as a mini-batch update (eq. lsqA_sto on column block k for +(k+1), the
 * analogous update of B on row block k for -(k+1)) with the context's eta and momentum,
 * whatever its mode.  Does not advance the sweep counter.  Arguments and errors as for
 * nmd_als_block_sweep.
 */
int nmd_run_steps(nmd_ctx* ctx, float* W, float* H, const int32_t* steps, int32_t n_steps,
                  void* hip_stream);

/*
 * nmd_rectified_contraction - the dense product of a step on its own: Y = max(0, A B^T) B, the
 * rectified low-rank matrix S-hat of eq. rectify contracted with the panel (the dense term of
 * Delta B in eqs. updateD and spLsqA), for device row-major A (rows x r), B (blk x r) and Y
 * (rows x r, overwritten).  The L tile is never written to memory (the fused kernel of Sec.
 * 4.2), and the second product is skipped on every slice of 16 rows x 4 panel rows where S-hat
 * is zero (Sec. 4.3).  r must be 16, 32, 48, 64 or a multiple of 64 up to 512; rows >= 1 and
 * <= 2^31 - 1, blk >= 1.  Padding columns of A and B must hold zeros.  One fp32 accumulation
 * over all of B.  Asynchronous on hip_stream; allocates nothing.  NMD_EINVAL on bad arguments,
 * NMD_EDEVICE if the launch fails.
 */
int nmd_rectified_contraction(const float* A, int64_t rows, const float* B, int64_t blk,
                              int32_t r, float* Y, void* hip_stream);

/*
 * nmd_rectified_contraction_bf16x3 - the same product Y = max(0, A B^T) B with BOTH products on
 * bf16 MFMA of two-term operand splits (x = bf16(x) + bf16(x - bf16(x)), three products each,
 * fp32 accumulation): the counterpart, for a dense max(0, A B^T), of the paper's TF32 fused
 * kernels (Sec. 4.2, kernel throughput table).  Relative error of each output about 2^-16 of
 * the sum of the magnitudes of its terms.  A: device rows x r, B: device blk x r, Y: device
 * rows x r (all fp32 row-major), r in {16, 32, 64, 128, 256, 512}.  work: caller-owned device
 * workspace of nmd_bf16x3_workspace_floats(blk, r) floats, overwritten with the split panel
 * (row-major and, at r <= 128, transposed copies).  Asynchronous on hip_stream; allocates
 * nothing.  NMD_EINVAL on NULL
 * pointers, another r or bad sizes, NMD_EDEVICE if a launch fails.
 */
int nmd_rectified_contraction_bf16x3(const float* A, int64_t rows, const float* B, int64_t blk,
                                     int32_t r, float* work, float* Y, void* hip_stream);

/*
 * nmd_rectified_contraction_bf16x3_noalloc - nmd_rectified_contraction_bf16x3 for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same product with the same kernels and results, but the split
 * panel goes to a static workspace of 4 Mi floats (16 MiB) that the library keeps on every
 * device it runs on until the process ends, so no `work` argument is taken.  A, B, Y, r and
 * the errors as for nmd_rectified_contraction_bf16x3; a panel whose
 * nmd_bf16x3_workspace_floats(blk, r) exceeds 4 Mi floats (blk > 8192 at r = 512, > 16384 at
 * r = 256) is rejected with NMD_EINVAL before any launch.  Calls no allocating routine.  All
 * calls on one device share its workspace: calls that overlap on one device (other streams,
 * other threads) race and must be ordered by the caller.  Asynchronous on hip_stream.
 */
int nmd_rectified_contraction_bf16x3_noalloc(const float* A, int64_t rows, const float* B,
                                             int64_t blk, int32_t r, float* Y, void* hip_stream);

/*
 * nmd_bf16x3_workspace_floats - floats of workspace nmd_rectified_contraction_bf16x3 needs for
 * a blk-row panel at rank r: blk r + 32 ceil(blk / 32) max(r, 32) for r <= 128, blk r for
 * r = 256 and 512 (whose kernels read the row-major copy transposed in LDS).  -1 if blk < 1 or
 * r is not one of 16, 32, 64, 128, 256, 512.
 */
int64_t nmd_bf16x3_workspace_floats(int64_t blk, int32_t r);

/*
 * nmd_get_dense_blocks - how much of the second product of the dense contraction the sweeps
 * ran, since the context was created or last reset here.  The second product is organised in
 * slices of 16 rows x 4 panel rows of max(0, L) (Sec. 4.3: S-hat is sparse): a slice with no
 * positive entry is skipped and the others run their own MFMAs; at r_p = 256 and 512 the
 * second product instead runs per quad-column (4 rows x 1 panel row) holding a positive entry.
 * *run = slices that ran whole, *total = slices examined, *entries = positive entries taken
 * by quad-columns (r_p = 256, 512); the second product's useful work is run/total of its dense
 * count plus 2 r flops per entry.  Synchronises the device.
 * reset != 0 clears all three after reading.  Any output pointer may be NULL.
 */
int nmd_get_dense_blocks(nmd_ctx* ctx, int64_t* run, int64_t* total, int64_t* entries,
                         int32_t reset);

/*
 * nmd_get_kernel_timing - with NMD_FLAG_TIMING set, the summed device time (HIP events on the
 * stream the work ran on) and launch count of one kernel class since the last reset of the
 * timers, plus the algorithmic work of those launches.  kernel: 0 = fused dense contraction
 * (flops = 4 rows blk r per launch), 1 = sparse correction (bytes = algorithmic HBM bytes; at
 * r_p >= 320 it runs on its own stream, beside the contraction, and this is its time there),
 * 2 = Gram matrices and inverses (side stream; one entry per run of same-side steps), 3 = solve
 * and update, 4 = the time the caller's stream waited for the side stream before an update
 * (zero when the solve was ready; no work).  Synchronises the recorded events.
 * reset != 0 clears the timers after reading.  Any output pointer may be NULL.
 */
int nmd_get_kernel_timing(nmd_ctx* ctx, int32_t kernel, double* total_ms, int64_t* launches,
                          double* flops, double* bytes, int32_t reset);

#ifdef __cplusplus
}
#endif

#endif /* NMD_H */
