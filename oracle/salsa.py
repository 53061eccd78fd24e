"""Stochastic alternating least squares for subzero matrix completion, in plain fp64 numpy.

Notation follows the paper: S (m x n, sparse, nonnegative), L = A B^T with A (m x r) and
B (n x r) (eq. ABt); in the GPU library's terms A = W and B = H^T.

The routines below take the algorithm's steps in the paper's order and form the dense
matrices L, S-hat and Delta explicitly, one tile of rows at a time (at most `row_chunk` rows
by one block of columns), so that no m x n matrix is held (Sec. 4.1, parallel least squares).

Readings of the paper used here (each is also listed in the design notes):
  * eq. Delta_par and eq. Delta_sto print 1_S o (S - S_hat - A B^T); eq. updateD prints
    1_S o (S + S_hat - A B^T).  Substituting eq. updateZ into eq. Delta gives Delta = S - L on
    the nonzeros of S, which is the "+" form, so that form is used everywhere.
  * The superscript J in eq. Delta_sto restricts to the columns in J.
  * Momentum (Sec. 4.1: a heavy-ball term, gamma times the last step taken): heavy ball,
    V <- gamma V + eta Delta_{:J} B_J [B_J^T B_J]^{-1}, A <- A + V, one buffer per factor,
    zero at the start.
  * The r x r systems are solved by a Cholesky factorisation of the Gram matrix.
"""

from __future__ import annotations

import numpy as np
import scipy.linalg as sla
import scipy.sparse as sp

from . import partition, schedule


# --------------------------------------------------------------------------------------------
# Elementwise definitions (Sec. 3.1 and 3.2)
# --------------------------------------------------------------------------------------------

def rectify(L):
    """S-hat = max(0, L) (eq. rectify)."""
    return np.maximum(0.0, L)


def z_update(S, L):
    """Z = S where S > 0, else L - S-hat (eq. updateZ); S and L dense."""
    return np.where(S > 0, S, L - rectify(L))


def delta_update(S, A, B):
    """Delta = 1_S o (S + S-hat - A B^T) - S-hat (eq. updateD), dense S."""
    L = A @ B.T
    Shat = rectify(L)
    return (S > 0) * (S + Shat - L) - Shat


def aux_objective_dense(S, L):
    """||Z - L||_F / ||S||_F with Z from eq. updateZ (eq. auxCost at its optimal Z)."""
    Z = z_update(S, L)
    return np.linalg.norm(Z - L) / np.linalg.norm(S)


def squared_loss_dense(S, L):
    """sum over zeros of max(0, L)^2 plus sum over nonzeros of (S - L)^2 (eq. SLloss)."""
    pos = S > 0
    return float(np.sum(np.where(pos, 0.0, rectify(L) ** 2)) + np.sum(np.where(pos, (S - L) ** 2, 0.0)))


def rmse_dense(S, Shat):
    """||S - S-hat||_F / ||S||_F (eq. RMSE)."""
    return np.linalg.norm(S - Shat) / np.linalg.norm(S)


def wjd_dense(S, Shat):
    """1 - sum min(S, S-hat) / sum max(S, S-hat) (eq. WJD)."""
    return 1.0 - np.sum(np.minimum(S, Shat)) / np.sum(np.maximum(S, Shat))


# --------------------------------------------------------------------------------------------
# Sparse inputs
# --------------------------------------------------------------------------------------------

def csr_matrix(m, n, row_ptr, col, val):
    """S as a float64 scipy CSR matrix; explicit zeros are dropped (the mask is S_ij > 0)."""
    S = sp.csr_matrix((np.asarray(val, dtype=np.float64), np.asarray(col, dtype=np.int64),
                       np.asarray(row_ptr, dtype=np.int64)), shape=(m, n))
    S.eliminate_zeros()
    return S


class State:
    """Factors A (m x r), B (n x r), their momentum buffers and the sweep counter."""

    def __init__(self, W, H):
        self.A = np.array(W, dtype=np.float64)          # A = W
        self.B = np.array(H, dtype=np.float64).T.copy()  # B = H^T
        self.VA = np.zeros_like(self.A)
        self.VB = np.zeros_like(self.B)
        self.t = 0

    @property
    def W(self):
        return self.A

    @property
    def H(self):
        return self.B.T


# --------------------------------------------------------------------------------------------
# One factor update from one block of the other factor
# --------------------------------------------------------------------------------------------

def _gram_factor(PJ):
    G = PJ.T @ PJ
    return sla.cho_factor(G, lower=True, check_finite=True)


def factor_step(S_rows, X, P, j0, j1, eta, gamma, V, row_chunk=4096, rows=None):
    """Stochastic least-squares update of X from the columns [j0, j1) of S_rows (eqs. Shat_sto,
    Delta_sto, lsqA_sto, plus momentum).

    S_rows is the sparse matrix whose rows index X (S itself when X = A, S^T when X = B), P the
    other factor.  Row tiles follow the blockwise form of eq. lsqA_par.  Returns the new X and
    V; when `rows` is given only those rows are computed and returned (X[rows], V[rows])."""
    PJ = P[j0:j1]
    cf = _gram_factor(PJ)                                 # B_J^T B_J = L L^T
    SJ = S_rows[:, j0:j1].tocsr()
    idx = np.arange(X.shape[0]) if rows is None else np.asarray(rows)
    U = np.empty((idx.size, X.shape[1]))
    for s in range(0, idx.size, row_chunk):
        I = idx[s:s + row_chunk]
        L = X[I] @ PJ.T                                   # eq. ABt on the tile
        Shat = rectify(L)                                 # eq. Shat_sto
        Sd = SJ[I].toarray()
        Delta = (Sd > 0) * (Sd + Shat - L) - Shat         # eq. Delta_sto ("+" reading)
        U[s:s + row_chunk] = Delta @ PJ
    step = sla.cho_solve(cf, U.T).T                       # Delta_{:J} B_J [B_J^T B_J]^{-1}
    Vn = gamma * V[idx] + eta * step
    return X[idx] + Vn, Vn


def w_step(S, st: State, j0, j1, eta, gamma, row_chunk=4096):
    """Update A from the column mini-batch J = [j0, j1) (eq. lsqA_sto with momentum)."""
    st.A, st.VA = factor_step(S, st.A, st.B, j0, j1, eta, gamma, st.VA, row_chunk)


def h_step(ST, st: State, i0, i1, eta, gamma, row_chunk=4096):
    """Update B from the row mini-batch I = [i0, i1): the same update on S^T (the analogous
    update for block rows of B, Sec. 4.1)."""
    st.B, st.VB = factor_step(ST, st.B, st.A, i0, i1, eta, gamma, st.VB, row_chunk)


def run_steps(S, ST, st: State, steps, block_m, block_n, eta, gamma, row_chunk=4096):
    """Execute encoded steps: +(k+1) = W-step on column block k, -(k+1) = H-step on row
    block k."""
    m, n = S.shape
    rb = partition.bounds(m, block_m)
    cb = partition.bounds(n, block_n)
    for code in steps:
        if code > 0:
            k = code - 1
            w_step(S, st, cb[k], cb[k + 1], eta, gamma, row_chunk)
        else:
            k = -code - 1
            h_step(ST, st, rb[k], rb[k + 1], eta, gamma, row_chunk)


def sweep(S, ST, st: State, block_m, block_n, seed, mode="stochastic", eta=1.0, gamma=0.0,
          row_chunk=4096):
    """One sweep (epoch).  Stochastic: the seeded interleaved list of W- and H-steps.
    Deterministic: the exact least-squares half-steps A <- A + Delta B (B^T B)^{-1} over all
    columns (eq. spLsqA), then B <- B + Delta^T A (A^T A)^{-1} over all rows (eq. spLsqB),
    each evaluated in row tiles (eq. lsqA_par); eta and gamma apply as in the stochastic
    update (eta = 1, gamma = 0 gives the plain half-steps)."""
    m, n = S.shape
    if mode == "stochastic":
        R = partition.num_blocks(m, block_m)
        C = partition.num_blocks(n, block_n)
        steps = schedule.sweep_schedule(seed, st.t, R, C, True)
        run_steps(S, ST, st, steps, block_m, block_n, eta, gamma, row_chunk)
    else:
        w_step(S, st, 0, n, eta, gamma, row_chunk)
        h_step(ST, st, 0, m, eta, gamma, row_chunk)
    st.t += 1


# --------------------------------------------------------------------------------------------
# Objective and metrics, tiled over rows
# --------------------------------------------------------------------------------------------

def objective(S, W, H, row_chunk=2048):
    """f = sqrt(sum_{S=0} max(0,L)^2 + sum_{S>0} (S-L)^2) / ||S||_F, L = W H (eq. auxCost with Z
    eliminated by eq. SLloss)."""
    W = np.asarray(W, dtype=np.float64)
    H = np.asarray(H, dtype=np.float64)
    total = 0.0
    for r0 in range(0, S.shape[0], row_chunk):
        L = W[r0:r0 + row_chunk] @ H
        Sd = S[r0:r0 + row_chunk].toarray()
        pos = Sd > 0
        total += float(np.sum(np.where(pos, (Sd - L) ** 2, rectify(L) ** 2)))
    return float(np.sqrt(total) / sp.linalg.norm(S))


def rmse(S, W, H, row_chunk=2048):
    W = np.asarray(W, dtype=np.float64)
    H = np.asarray(H, dtype=np.float64)
    num = 0.0
    for r0 in range(0, S.shape[0], row_chunk):
        Sd = S[r0:r0 + row_chunk].toarray()
        num += float(np.sum((Sd - rectify(W[r0:r0 + row_chunk] @ H)) ** 2))
    return float(np.sqrt(num) / sp.linalg.norm(S))


def wjd(S, W, H, row_chunk=2048):
    W = np.asarray(W, dtype=np.float64)
    H = np.asarray(H, dtype=np.float64)
    lo = hi = 0.0
    for r0 in range(0, S.shape[0], row_chunk):
        Sd = S[r0:r0 + row_chunk].toarray()
        Sh = rectify(W[r0:r0 + row_chunk] @ H)
        lo += float(np.sum(np.minimum(Sd, Sh)))
        hi += float(np.sum(np.maximum(Sd, Sh)))
    return 1.0 - lo / hi


# --------------------------------------------------------------------------------------------
# The dense contraction on its own (the product of the fused kernel, Sec. 4.2)
# --------------------------------------------------------------------------------------------

def clamped_contraction(A, BJ):
    """min(0, A B_J^T) B_J: the dense part of Z_{:,J} B_J on the zeros of S."""
    A = np.asarray(A, dtype=np.float64)
    BJ = np.asarray(BJ, dtype=np.float64)
    return np.minimum(0.0, A @ BJ.T) @ BJ


def rectified_contraction(A, BJ):
    """max(0, A B_J^T) B_J: the rectified low-rank matrix of eq. rectify times the panel, the
    dense term of Delta_{:,J} B_J (eq. updateD off the nonzeros of S, contracted as in
    eq. spLsqA)."""
    A = np.asarray(A, dtype=np.float64)
    BJ = np.asarray(BJ, dtype=np.float64)
    return rectify(A @ BJ.T) @ BJ


def zb_product(S_rows, X, P, j0, j1, rows=None):
    """Z_{I,J} P_J for the rows I of X (all rows by default): the right-hand side of the
    least-squares update in Z form (eq. lsqA restricted to the columns J)."""
    X = np.asarray(X, dtype=np.float64)
    P = np.asarray(P, dtype=np.float64)
    idx = np.arange(X.shape[0]) if rows is None else np.asarray(rows)
    PJ = P[j0:j1]
    L = X[idx] @ PJ.T
    Sd = S_rows[:, j0:j1].tocsr()[idx].toarray()
    return z_update(Sd, L) @ PJ


# --------------------------------------------------------------------------------------------
# Step-size safeguard (a reading of Sec. 7 and the appendix on experimental settings)
# --------------------------------------------------------------------------------------------

def guarded_sweeps(S, ST, st: State, block_m, block_n, seed, n_sweeps, mode="stochastic",
                   eta=1.0, gamma=0.0, tol=0.0, eta_min=0.0, row_chunk=4096):
    """n_sweeps accepted sweeps under a step-size safeguard.

    The paper notes that the stochastic updates can diverge when the step size is too large
    (Sec. 7) and lowers the step size for the models that need it (appendix on experimental
    settings, hyperparameter table); it gives no automatic rule.  The rule read here: after each
    sweep the objective is evaluated; a sweep that leaves it above (1 + tol) times its value
    before the sweep (or not finite) is undone -- both factors and the sweep counter return to
    their values before the sweep -- the momentum buffers are cleared (a restart of the heavy
    ball), the step size is halved, and the sweep is run again with the same block order.  The
    comparison is made on the squared objective, f_new^2 > (1 + tol)^2 f_old^2.  Halving stops
    with a ValueError once the step size would fall below eta_min.

    Returns (eta, f, rejected): the step size in force at the end, the objective before the
    first sweep and after each accepted sweep (n_sweeps + 1 values), and the list of
    (sweep counter, step size, objective) of each rejected attempt."""
    f_prev = objective(S, st.W, st.H)
    fs = [f_prev]
    rejected = []
    done = 0
    while done < n_sweeps:
        saved = (st.A.copy(), st.B.copy(), st.t)
        sweep(S, ST, st, block_m, block_n, seed, mode, eta, gamma, row_chunk)
        f = objective(S, st.W, st.H)
        if not (f * f <= (1.0 + tol) ** 2 * f_prev * f_prev):
            rejected.append((saved[2], eta, f))
            st.A, st.B, st.t = saved
            st.VA = np.zeros_like(st.A)
            st.VB = np.zeros_like(st.B)
            eta = 0.5 * eta
            if eta < eta_min:
                raise ValueError("step size fell below eta_min")
            continue
        f_prev = f
        fs.append(f)
        done += 1
    return eta, fs, rejected
