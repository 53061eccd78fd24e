"""Pins of the fp64 oracle against what the paper and the mathematics fix (CPU only).

Each test names the passage it checks.  None of them re-types an oracle formula and compares
the oracle with itself: they use brute force, closed-form completions from Sec. 2, textbook
least squares, or invariants proved in the paper.
"""

import math

import numpy as np
import pytest
import scipy.sparse as sp

from oracle import partition, salsa
from workloads import gen


def _rand_problem(m, n, r, density, seed, sign_init=True):
    row_ptr, col, val = gen.random_sparse(m, n, density, seed)
    S = salsa.csr_matrix(m, n, row_ptr, col, val)
    if sign_init:
        W, H = gen.sign_constrained_init(m, n, r, float(val.mean()), seed + 7)
    else:
        W, H = gen.gaussian_init(m, n, r, 0.5, seed + 7)
    return S, W.astype(np.float64), H.astype(np.float64)


def _exact_state_sweep(S, W, H, mode="deterministic", block=(7, 5)):
    st = salsa.State(W, H)
    ST = S.T.tocsr()
    salsa.sweep(S, ST, st, block[0], block[1], seed=3, mode=mode)
    return st


# ---------------------------------------------------------------------------- P1: Z-update
def test_z_update_is_elementwise_constrained_argmin():
    """eq. updateZ: for fixed L, Z minimises ||Z - L|| subject to S = max(0, Z) (Sec. 3.2).
    Brute force over a grid of candidates plus the analytic candidates {S_ij, L_ij, 0}."""
    rng = np.random.default_rng(11)
    grid = np.linspace(-4.0, 4.0, 10001)
    for _ in range(25):
        m, n = rng.integers(1, 7, 2)
        S = np.where(rng.random((m, n)) < 0.4, np.round(rng.uniform(0.25, 3.0, (m, n)), 2), 0.0)
        L = np.round(rng.uniform(-3.0, 3.0, (m, n)), 3)
        Z = salsa.z_update(S, L)
        for i in range(m):
            for j in range(n):
                cand = np.concatenate([grid, [S[i, j], L[i, j], 0.0]])
                feas = cand[np.maximum(0.0, cand) == S[i, j]]
                best = feas[np.argmin((feas - L[i, j]) ** 2)]
                assert best == Z[i, j]
                assert np.maximum(0.0, Z[i, j]) == S[i, j]


# ------------------------------------------------------------------- P2 / P11: LS update forms
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_stochastic_step_equals_textbook_least_squares(seed):
    """eq. lsqA_sto with eta = 1 and no momentum is the exact least-squares fit of the columns
    J of Z (eq. updateZ) by A B_J^T: compare with numpy.linalg.lstsq (Sec. 3.2, eq. lsqA)."""
    m, n, r = 37, 29, 4
    S, W, H = _rand_problem(m, n, r, 0.2, seed, sign_init=(seed != 2))
    A, B = W, H.T
    j0, j1 = 5, 23
    Sd = S.toarray()
    Z = salsa.z_update(Sd[:, j0:j1], A @ B[j0:j1].T)
    X_ls = np.linalg.lstsq(B[j0:j1], Z.T, rcond=None)[0].T
    X, V = salsa.factor_step(S, A, B, j0, j1, 1.0, 0.0, np.zeros_like(A))
    np.testing.assert_allclose(X, X_ls, rtol=1e-10, atol=1e-12 * np.abs(X_ls).max())
    np.testing.assert_allclose(V, X_ls - A, rtol=1e-9, atol=1e-12 * np.abs(X_ls).max())


def test_delta_form_matches_z_form():
    """eq. Delta with Z from eq. updateZ equals eq. updateD with the '+ S_hat' sign, i.e. the
    printed '- S_hat' of eqs. Delta_par/Delta_sto is a typo (the '+' reading)."""
    rng = np.random.default_rng(5)
    m, n, r = 23, 31, 5
    S = np.where(rng.random((m, n)) < 0.3, rng.uniform(0.1, 2.0, (m, n)), 0.0)
    A = rng.normal(size=(m, r))
    B = rng.normal(size=(n, r))
    L = A @ B.T
    np.testing.assert_allclose(salsa.delta_update(S, A, B), salsa.z_update(S, L) - L, atol=1e-13)
    minus_form = (S > 0) * (S - salsa.rectify(L) - L) - salsa.rectify(L)
    assert np.abs(minus_form - (salsa.z_update(S, L) - L)).max() > 1e-3


# ------------------------------------------------------------------- P3: monotone decrease
@pytest.mark.parametrize("case", ["config1_small", "identity256", "random_gauss"])
def test_deterministic_half_steps_never_increase_objective(case):
    """Alternating minimisation decreases the objective monotonically (Sec. 3.2); checked
    after every half-step for 20 sweeps."""
    if case == "config1_small":
        row_ptr, col, val, _ = gen.planted(300, 260, 8, 0.05, 1)
        m, n, r = 300, 260, 8
        W, H = gen.sign_constrained_init(m, n, r, float(val.mean()), 1001)
    elif case == "identity256":
        m = n = 256
        r = 3
        row_ptr, col, val = gen.identity(n)
        W, H = gen.gaussian_init(m, n, r, 0.1, 1002)
    else:
        m, n, r = 120, 90, 6
        row_ptr, col, val = gen.random_sparse(m, n, 0.1, 3)
        W, H = gen.gaussian_init(m, n, r, 0.5, 1003)
    S = salsa.csr_matrix(m, n, row_ptr, col, val)
    ST = S.T.tocsr()
    st = salsa.State(W, H)
    f = salsa.objective(S, st.W, st.H)
    for _ in range(20):
        salsa.w_step(S, st, 0, n, 1.0, 0.0)
        f1 = salsa.objective(S, st.W, st.H)
        assert f1 <= f * (1 + 1e-12)
        salsa.h_step(ST, st, 0, m, 1.0, 0.0)
        f2 = salsa.objective(S, st.W, st.H)
        assert f2 <= f1 * (1 + 1e-12)
        f = f2


# ------------------------------------------------- P4: identity and its rank-3 completion
@pytest.mark.parametrize("n", [5, 64, 256])
def test_identity_completion_closed_form(n):
    """Corollary 1, eq. Omega: Omega_ij = (cos(2 pi (i-j)/n) - cos(2 pi/n)) / (1 - cos(2 pi/n))
    has rank 3 and max(0, Omega) = I_n; the objective vanishes there."""
    W, H = gen.identity_exact_factors(n)
    i, j = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    c = math.cos(2 * math.pi / n)
    Omega = (np.cos(2 * math.pi * (i - j) / n) - c) / (1 - c)
    np.testing.assert_allclose(W @ H, Omega, atol=1e-9 * n * n)
    sv = np.linalg.svd(Omega, compute_uv=False)
    assert np.sum(sv > 1e-9 * sv[0]) == 3
    np.testing.assert_allclose(np.maximum(0, Omega), np.eye(n), atol=1e-9)
    S = salsa.csr_matrix(n, n, *gen.identity(n))
    assert salsa.objective(S, W, H) < 1e-9


def test_identity_completion_is_als_fixed_point_and_permutation():
    """The exact completion is a fixed point of the deterministic sweep (Z = L there), and a
    permuted identity P has the completion P Omega (Corollary 1)."""
    n = 512
    W, H = gen.identity_exact_factors(n)
    S = salsa.csr_matrix(n, n, *gen.identity(n))
    st = _exact_state_sweep(S, W, H)
    assert np.linalg.norm(st.W - W) / np.linalg.norm(W) < 1e-9
    assert np.linalg.norm(st.H - H) / np.linalg.norm(H) < 1e-9
    perm = np.random.default_rng(0).permutation(n)
    P = sp.csr_matrix((np.ones(n), (np.arange(n), perm)), shape=(n, n))
    # row i of P has its one in column perm[i]: P = max(0, W[perm] H)
    assert salsa.objective(P, W[perm], H) < 1e-9


# ------------------------------------------------------------ P5: ring signless Laplacian
@pytest.mark.parametrize("delta", [0.25, 0.5])
def test_ring_completion(delta):
    """Prop. 4: with tau (eq. tau) and r^2 (eq. r2), the thresholded similarities of
    equispaced planar points (eqs. ringvecs, tsm-sym) reproduce eq. ring; Prop. 1 turns them
    into a rank-3 completion, a zero of the objective and a fixed point of the sweep."""
    n = 64
    c = math.cos(2 * math.pi / n)
    tau = (c - delta) / (1 - delta)
    r2 = (1 - delta) / (1 - c)
    th = 2 * math.pi * np.arange(n) / n
    alpha = math.sqrt(r2) * np.stack([np.cos(th), np.sin(th)], 1)
    nrm = np.linalg.norm(alpha, axis=1)
    a = np.concatenate([alpha, (tau * nrm)[:, None]], 1)
    b = np.concatenate([alpha, (-nrm)[:, None]], 1)
    S = np.zeros((n, n))
    for i in range(n):
        S[i, i] = 1.0
        S[i, (i + 1) % n] = delta
        S[i, (i - 1) % n] = delta
    np.testing.assert_allclose(np.maximum(0, a @ b.T), S, atol=1e-12)
    Ssp = sp.csr_matrix(S)
    assert salsa.objective(Ssp, a, b.T) < 1e-9
    st = _exact_state_sweep(Ssp, a, b.T)
    assert np.linalg.norm(st.W - a) / np.linalg.norm(a) < 1e-8


# ------------------------------------------------------ P6: thresholded similarity matrix
def test_thresholded_similarity_completion():
    """Prop. 1: a_i = (alpha_i, tau |alpha_i|), b_j = (beta_j, -|beta_j|) complete eq. tsm
    with rank d + 1; the objective is 0 and both update modes leave the factors unchanged."""
    rng = np.random.default_rng(3)
    m, n, d, tau = 90, 70, 4, 0.55
    al = rng.normal(size=(m, d))
    be = rng.normal(size=(n, d))
    na = np.linalg.norm(al, axis=1)
    nb = np.linalg.norm(be, axis=1)
    S = np.maximum(0.0, al @ be.T - tau * np.outer(na, nb))
    a = np.concatenate([al, (tau * na)[:, None]], 1)
    b = np.concatenate([be, (-nb)[:, None]], 1)
    np.testing.assert_allclose(np.maximum(0, a @ b.T), S, atol=1e-12)
    Ssp = sp.csr_matrix(S)
    assert salsa.objective(Ssp, a, b.T) < 1e-10
    for mode in ("deterministic", "stochastic"):
        st = salsa.State(a, b.T)
        salsa.sweep(Ssp, Ssp.T.tocsr(), st, 30, 25, seed=9, mode=mode, eta=1.0, gamma=0.9)
        assert np.linalg.norm(st.W - a) / np.linalg.norm(a) < 1e-9
        assert np.linalg.norm(st.H - b.T) / np.linalg.norm(b) < 1e-9


# ---------------------------------------------------------------------- P7: hypercube graph
def test_hypercube_completion():
    """Prop. 5: alpha_i = rho v_i with rho^2 = (1 - delta)/2 and tau = 1 - (2/d)(1 - delta)^-1
    reproduce eq. hypercube (1 on the diagonal, delta between neighbours) with rank d + 1."""
    d, delta = 8, 0.06
    V = np.array([[1.0 if (k >> b) & 1 else -1.0 for b in range(d)] for k in range(2 ** d)])
    rho = math.sqrt((1 - delta) / 2)
    tau = 1 - (2.0 / d) / (1 - delta)
    al = rho * V
    nrm = np.linalg.norm(al, axis=1)
    a = np.concatenate([al, (tau * nrm)[:, None]], 1)
    b = np.concatenate([al, (-nrm)[:, None]], 1)
    ham = (V[:, None, :] != V[None, :, :]).sum(-1)
    S = np.where(ham == 0, 1.0, np.where(ham == 1, delta, 0.0))
    np.testing.assert_allclose(np.maximum(0, a @ b.T), S, atol=1e-12)
    assert salsa.objective(sp.csr_matrix(S), a, b.T) < 1e-10


# ----------------------------------------------------------- P8: block-diagonal matrices
@pytest.mark.parametrize("k,m,n,density", [(3, 3, 4, 1.0), (5, 4, 6, 0.6), (8, 3, 5, 0.8)])
def test_block_diagonal_completion(k, m, n, density):
    """Lemma 1 (eq. blocks, eq. hadamard): for k equal m x n nonnegative blocks S_b, the matrix
    L = (1_k kron [S_1 ... S_k]) hadamard (Omega kron 1_m 1_n^T), with Omega the completion of
    I_k (eq. Omega), satisfies max(0, L) = S and has rank <= 3m, independent of k.  Rank-3m
    factors W[(a,i),(p,q)] = [i = p] w_a[q], H[(p,q),(b,j)] = S_b[p,j] h_b[q] reproduce L, give
    objective 0, and are a fixed point of the deterministic sweep.  (The printed all-ones
    factor 1_m must be 1_k for the sizes km x kn to agree.)"""
    rng = np.random.default_rng(k * 100 + m * 10 + n)
    blocks = [np.where(rng.random((m, n)) < density, rng.uniform(0.2, 2.0, (m, n)), 0.0)
              for _ in range(k)]
    for Sb in blocks:  # every row and column of a block keeps a positive entry
        Sb[np.arange(m), np.arange(m) % n] = rng.uniform(0.5, 1.5, m)
        Sb[np.arange(n) % m, np.arange(n)] = rng.uniform(0.5, 1.5, n)
    S = np.zeros((k * m, k * n))
    for b, Sb in enumerate(blocks):
        S[b * m:(b + 1) * m, b * n:(b + 1) * n] = Sb
    # eq. Omega for I_k
    c = math.cos(2 * math.pi / k)
    th = 2 * math.pi * np.arange(k) / k
    Wo = np.stack([np.cos(th), np.sin(th), np.ones(k)], axis=1)
    Ho = np.stack([np.cos(th), np.sin(th), -c * np.ones(k)], axis=0) / (1 - c)
    Omega = Wo @ Ho
    L = np.kron(np.ones((k, 1)), np.hstack(blocks)) * np.kron(Omega, np.ones((m, n)))
    np.testing.assert_allclose(np.maximum(0.0, L), S, atol=1e-12)
    sv = np.linalg.svd(L, compute_uv=False)
    assert np.sum(sv > 1e-10 * sv[0]) <= 3 * m
    W = np.zeros((k * m, 3 * m))
    H = np.zeros((3 * m, k * n))
    for a in range(k):
        for i in range(m):
            W[a * m + i, i * 3:(i + 1) * 3] = Wo[a]
    for b, Sb in enumerate(blocks):
        for pidx in range(m):
            for q in range(3):
                H[pidx * 3 + q, b * n:(b + 1) * n] = Sb[pidx] * Ho[q, b]
    np.testing.assert_allclose(W @ H, L, atol=1e-12)
    Ssp = sp.csr_matrix(S)
    assert salsa.objective(Ssp, W, H) < 1e-9
    st = _exact_state_sweep(Ssp, W, H, block=(k * m, k * n))
    assert np.linalg.norm(st.W @ st.H - L) / np.linalg.norm(L) < 1e-9


# --------------------------------------------------------------- P9 / P10: the objective
def test_objective_routes_agree_and_bound_rmse():
    """eq. SLloss (Z eliminated) equals eq. auxCost evaluated with the optimal Z, and by
    Prop. 9 the objective is never below the RMSE (eq. RMSE)."""
    rng = np.random.default_rng(8)
    for _ in range(10):
        m, n, r = rng.integers(3, 40, 3)
        S = np.where(rng.random((m, n)) < 0.2, rng.uniform(0.1, 3.0, (m, n)), 0.0)
        S[0, 0] = 1.0
        L = rng.normal(size=(m, r)) @ rng.normal(size=(r, n))
        f_aux = salsa.aux_objective_dense(S, L)
        f_sl = math.sqrt(salsa.squared_loss_dense(S, L)) / np.linalg.norm(S)
        assert abs(f_aux - f_sl) <= 1e-12 * max(1.0, f_aux)
        assert f_aux >= salsa.rmse_dense(S, np.maximum(0, L)) - 1e-15
        A = rng.normal(size=(m, r))
        Bt = rng.normal(size=(r, n))
        Ssp = sp.csr_matrix(S)
        for chunk in (1, 7, 4096):
            f_tiled = salsa.objective(Ssp, A, Bt, row_chunk=chunk)
            assert abs(f_tiled - salsa.aux_objective_dense(S, A @ Bt)) <= 1e-12 * max(1, f_tiled)
        assert salsa.objective(Ssp, A, Bt) >= salsa.rmse(Ssp, A, Bt) - 1e-15
    # metrics are calibrated so that the all-zero approximation scores one (Sec. 3.1)
    S = np.where(rng.random((9, 8)) < 0.3, 1.5, 0.0)
    S[1, 1] = 2.0
    assert abs(salsa.rmse_dense(S, np.zeros_like(S)) - 1.0) < 1e-15
    assert abs(salsa.wjd_dense(S, np.zeros_like(S)) - 1.0) < 1e-15
    assert salsa.wjd_dense(S, S) == 0.0


# ------------------------------------------------------------------- P12: kernel algebra
def test_clamped_contraction_identity():
    """min(0, L) B_J = A (B_J^T B_J) - max(0, L) B_J, relating the clamped contraction to the
    paper's fused product max(0, A B^T)(B^+)^T (eq. kernel)."""
    rng = np.random.default_rng(4)
    A = rng.normal(size=(50, 12))
    BJ = rng.normal(size=(33, 12))
    L = A @ BJ.T
    lhs = salsa.clamped_contraction(A, BJ)
    rhs = A @ (BJ.T @ BJ) - np.maximum(0, L) @ BJ
    np.testing.assert_allclose(lhs, rhs, atol=1e-11)
    # against a brute-force sum over j
    brute = np.zeros_like(A)
    for i in range(A.shape[0]):
        for j in range(BJ.shape[0]):
            brute[i] += min(0.0, float(A[i] @ BJ[j])) * BJ[j]
    np.testing.assert_allclose(lhs, brute, atol=1e-11)


def test_rectified_contraction_and_delta_form():
    """max(0, L) B_J by explicit loops, and the Delta form of the right-hand side that the
    update uses: Delta_{:,J} B_J = Z_{:,J} B_J - A (B_J^T B_J) (eq. Delta with Z from eq. updateZ)
    equals the sum over the nonzeros of (s - min(0, l)) b_j minus max(0, L) B_J."""
    rng = np.random.default_rng(7)
    m, n, r, j0, j1 = 10, 13, 4, 3, 11
    S = np.where(rng.random((m, n)) < 0.3, rng.uniform(0.2, 2.0, (m, n)), 0.0)
    A = rng.normal(size=(m, r))
    B = rng.normal(size=(n, r))
    BJ = B[j0:j1]
    rect = salsa.rectified_contraction(A, BJ)
    brute = np.zeros((m, r))
    for i in range(m):
        for j in range(BJ.shape[0]):
            brute[i] += max(0.0, float(A[i] @ BJ[j])) * BJ[j]
    np.testing.assert_allclose(rect, brute, atol=1e-12)
    corr = np.zeros((m, r))
    for i in range(m):
        for j in range(j0, j1):
            if S[i, j] > 0:
                corr[i] += (S[i, j] - min(0.0, float(A[i] @ B[j]))) * B[j]
    delta_b = salsa.zb_product(sp.csr_matrix(S), A, B, j0, j1) - A @ (BJ.T @ BJ)
    np.testing.assert_allclose(corr - rect, delta_b, atol=1e-11)
    # a sign-constrained pair (A > 0, B < 0) has S-hat = 0 (Sec. 4.3)
    assert not np.any(salsa.rectified_contraction(np.abs(A), -np.abs(BJ)))


def test_zb_product_brute_force():
    """Z_{:,J} B_J by explicit loops over eq. updateZ."""
    rng = np.random.default_rng(6)
    m, n, r = 9, 11, 3
    S = np.where(rng.random((m, n)) < 0.3, rng.uniform(0.2, 2.0, (m, n)), 0.0)
    A = rng.normal(size=(m, r))
    B = rng.normal(size=(n, r))
    out = salsa.zb_product(sp.csr_matrix(S), A, B, 2, 9)
    brute = np.zeros((m, r))
    for i in range(m):
        for j in range(2, 9):
            l = float(A[i] @ B[j])
            z = S[i, j] if S[i, j] > 0 else min(0.0, l)
            brute[i] += z * B[j]
    np.testing.assert_allclose(out, brute, atol=1e-12)


# ----------------------------------------------------- P13: stochastic vs deterministic
def test_one_block_stochastic_sweep_is_deterministic_sweep():
    """With a single row block and a single column block, eta = 1 and no momentum, the
    stochastic sweep performs exactly the two full least-squares half-steps; eta = 0 and no
    momentum leaves the factors unchanged (eq. lsqA_sto)."""
    m, n, r = 60, 45, 5
    S, W, H = _rand_problem(m, n, r, 0.15, 21)
    st_s = salsa.State(W, H)
    salsa.sweep(S, S.T.tocsr(), st_s, m, n, seed=4, mode="stochastic", eta=1.0, gamma=0.0)
    st_d = salsa.State(W, H)
    salsa.sweep(S, S.T.tocsr(), st_d, 7, 3, seed=4, mode="deterministic")
    np.testing.assert_allclose(st_s.A, st_d.A, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(st_s.B, st_d.B, rtol=1e-12, atol=1e-12)
    st_0 = salsa.State(W, H)
    salsa.sweep(S, S.T.tocsr(), st_0, 16, 16, seed=4, mode="stochastic", eta=0.0, gamma=0.0)
    assert np.array_equal(st_0.A, W) and np.array_equal(st_0.B, H.T)


def test_momentum_is_heavy_ball():
    """Heavy-ball momentum adds gamma times the last step taken (Sec. 4.1): two
    consecutive steps on the same block with gamma give A2 - A1 = gamma (A1 - A0) + eta D1."""
    m, n, r = 40, 30, 4
    S, W, H = _rand_problem(m, n, r, 0.2, 2)
    st = salsa.State(W, H)
    A0 = st.A.copy()
    salsa.w_step(S, st, 3, 20, 0.7, 0.9)
    A1 = st.A.copy()
    X1, _ = salsa.factor_step(S, A1, st.B, 3, 20, 1.0, 0.0, np.zeros_like(A1))
    salsa.w_step(S, st, 3, 20, 0.7, 0.9)
    np.testing.assert_allclose(st.A - A1, 0.9 * (A1 - A0) + 0.7 * (X1 - A1), atol=1e-12)


# ------------------------------------------------------------------ P14: block invariance
def test_row_tiling_and_blocks_do_not_change_results():
    """The parallel (row-blockwise) update eq. lsqA_par gives the same factors for any row
    tiling, and the deterministic sweep does not depend on the block sizes."""
    m, n, r = 70, 50, 6
    S, W, H = _rand_problem(m, n, r, 0.1, 13)
    ref = None
    for chunk, bm, bn in [(4096, 70, 50), (1, 7, 9), (13, 16, 50)]:
        st = salsa.State(W, H)
        salsa.sweep(S, S.T.tocsr(), st, bm, bn, seed=1, mode="deterministic", row_chunk=chunk)
        if ref is None:
            ref = st
        else:
            np.testing.assert_allclose(st.A, ref.A, rtol=1e-12, atol=1e-13)
            np.testing.assert_allclose(st.B, ref.B, rtol=1e-12, atol=1e-13)


def test_sampled_rows_match_full_step():
    """Row-sampled evaluation of a stochastic step (used for full-size checks) reproduces the
    full step on those rows."""
    m, n, r = 80, 60, 5
    S, W, H = _rand_problem(m, n, r, 0.1, 17)
    A, B = W, H.T
    V = np.random.default_rng(1).normal(size=A.shape) * 0.01
    X, Vn = salsa.factor_step(S, A, B, 10, 41, 0.8, 0.9, V)
    rows = np.array([0, 5, 79, 33])
    Xs, Vs = salsa.factor_step(S, A, B, 10, 41, 0.8, 0.9, V, rows=rows)
    np.testing.assert_allclose(Xs, X[rows], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(Vs, Vn[rows], rtol=1e-13, atol=1e-14)


def test_balanced_partition():
    for size, block in [(1000, 256), (139255, 8192), (50000, 8192), (500000, 16384), (5, 7)]:
        b = partition.bounds(size, block)
        K = len(b) - 1
        assert K == math.ceil(size / block)
        sizes = np.diff(b)
        assert b[0] == 0 and b[-1] == size
        assert sizes.max() <= block and sizes.max() - sizes.min() <= 1


# --------------------------------------------------- metrics: eq. RMSE and eq. WJD by value
def _hand_case():
    """S and L whose eq. RMSE and eq. WJD were worked out by hand (Sec. 3.1).

    S = [[2, 0, 0], [1, 3, 0]], L = [[1, 1, -2], [-1, 3, 1/2]], so S-hat = max(0, L) =
    [[1, 1, 0], [0, 3, 1/2]].
      S - S-hat = [[1, -1, 0], [1, 0, -1/2]]: squared sum 13/4; ||S||_F^2 = 14.
      RMSE = sqrt(13/56).
      sum min(S, S-hat) = 1 + 3 = 4; sum max(S, S-hat) = 2 + 1 + 1 + 3 + 1/2 = 15/2.
      WJD = 1 - 4 / (15/2) = 7/15.
    (A denominator of sum S = 6 would give 1/3, of sum S-hat = 11/2 would give 3/11.)"""
    S = np.array([[2.0, 0.0, 0.0], [1.0, 3.0, 0.0]])
    L = np.array([[1.0, 1.0, -2.0], [-1.0, 3.0, 0.5]])
    return S, L, math.sqrt(13.0 / 56.0), 7.0 / 15.0


def test_rmse_and_wjd_hand_computed_values():
    """eq. RMSE and eq. WJD on a 2 x 3 case computed by hand, for the dense metrics and for the
    row-tiled metrics over factors W H = L (W = I, H = L), at several row tilings."""
    S, L, rmse_ref, wjd_ref = _hand_case()
    Shat = np.maximum(0.0, L)
    assert abs(salsa.rmse_dense(S, Shat) - rmse_ref) < 1e-15
    assert abs(salsa.wjd_dense(S, Shat) - wjd_ref) < 1e-15
    Ssp = sp.csr_matrix(S)
    W = np.eye(2)
    for chunk in (1, 2, 2048):
        assert abs(salsa.rmse(Ssp, W, L, row_chunk=chunk) - rmse_ref) < 1e-15
        assert abs(salsa.wjd(Ssp, W, L, row_chunk=chunk) - wjd_ref) < 1e-15
    # the objective on the same case by hand: zeros of S contribute max(0, L)^2 = 1 and 1/4,
    # nonzeros (S - L)^2 = 1, 4, 0: total 25/4, so f = sqrt(25/56) (eqs. auxCost, SLloss)
    assert abs(salsa.objective(Ssp, W, L) - math.sqrt(25.0 / 56.0)) < 1e-15


@pytest.mark.parametrize("c", [0.25, 0.5, 1.0, 2.0, 5.0])
def test_rmse_and_wjd_of_a_scaled_reconstruction(c):
    """Closed forms for S-hat = c S (c > 0): every entry has min = min(1, c) S_ij and
    max = max(1, c) S_ij, so WJD = 1 - min(c, 1/c), and RMSE = |1 - c| (Sec. 3.1). Both
    vanish exactly at c = 1 (S = S-hat)."""
    rng = np.random.default_rng(8)
    S = np.where(rng.random((31, 17)) < 0.2, rng.uniform(0.5, 4.0, (31, 17)), 0.0)
    assert abs(salsa.wjd_dense(S, c * S) - (1.0 - min(c, 1.0 / c))) < 1e-14
    assert abs(salsa.rmse_dense(S, c * S) - abs(1.0 - c)) < 1e-14
    # tiled forms: L = c S written as W H with W = c I
    Ssp = sp.csr_matrix(S)
    for chunk in (1, 5, 2048):
        assert abs(salsa.wjd(Ssp, c * np.eye(31), S, row_chunk=chunk)
                   - (1.0 - min(c, 1.0 / c))) < 1e-14
        assert abs(salsa.rmse(Ssp, c * np.eye(31), S, row_chunk=chunk) - abs(1.0 - c)) < 1e-14


def test_tiled_metrics_match_dense_on_random_factors():
    """The row-tiled metrics equal the dense definitions for any tiling (Sec. 3.1), on random
    factors whose L has entries of both signs."""
    rng = np.random.default_rng(9)
    m, n, r = 23, 19, 3
    S = np.where(rng.random((m, n)) < 0.25, rng.uniform(0.1, 3.0, (m, n)), 0.0)
    W = rng.normal(size=(m, r))
    H = rng.normal(size=(r, n))
    Shat = np.maximum(0.0, W @ H)
    Ssp = sp.csr_matrix(S)
    for chunk in (1, 4, 7, 2048):
        assert abs(salsa.rmse(Ssp, W, H, row_chunk=chunk) - salsa.rmse_dense(S, Shat)) < 1e-14
        assert abs(salsa.wjd(Ssp, W, H, row_chunk=chunk) - salsa.wjd_dense(S, Shat)) < 1e-14


# ------------------------------------ step codes -> blocks (eqs. lsqA_sto and its H analogue)
def _projected_z(Sblk, Lblk):
    """Z entry by entry as the nearest point to L_ij of the set {z : max(0, z) = S_ij}: the
    single point S_ij when S_ij > 0, else the half-line z <= 0 (Sec. 3.2)."""
    Z = np.empty_like(Lblk)
    for i in range(Lblk.shape[0]):
        for j in range(Lblk.shape[1]):
            Z[i, j] = Sblk[i, j] if Sblk[i, j] > 0 else min(Lblk[i, j], 0.0)
    return Z


def test_step_codes_select_the_blocks_the_partition_names():
    """Each step code updates the factor and block it names: +k fits every row of A to the
    columns of column block k-1 (eq. lsqA_sto, eta = 1, no momentum), -k every row of B to
    the rows of row block k-1 (the analogous update of Sec. 4.1). m != n and the row and
    column blocks differ, so swapped bounds, a swapped sign convention or an off-by-one code
    would all fail. Expected values: numpy.linalg.lstsq on blocks sliced by hand from bounds
    worked out by hand from the balanced partition."""
    m, n, r = 13, 11, 2
    S, W, H = _rand_problem(m, n, r, 0.35, 31, sign_init=False)
    Sd = S.toarray()
    # balanced partition by hand: R = ceil(13/5) = 3 row blocks [floor(13k/3)], C = ceil(11/4)
    # = 3 column blocks [floor(11k/3)]
    rows = [0, 4, 8, 13]
    cols = [0, 3, 7, 11]
    assert list(partition.bounds(m, 5)) == rows and list(partition.bounds(n, 4)) == cols
    codes = [+2, -3, +1, -1, +3, -2, +2]
    st = salsa.State(W, H)
    A = W.copy()
    B = H.T.copy()
    for code in codes:
        salsa.run_steps(S, S.T.tocsr(), st, [code], 5, 4, 1.0, 0.0)
        if code > 0:
            j0, j1 = cols[code - 1], cols[code]
            Z = _projected_z(Sd[:, j0:j1], A @ B[j0:j1].T)
            A = np.linalg.lstsq(B[j0:j1], Z.T, rcond=None)[0].T
        else:
            i0, i1 = rows[-code - 1], rows[-code]
            Z = _projected_z(Sd[i0:i1, :], A[i0:i1] @ B.T)
            B = np.linalg.lstsq(A[i0:i1], Z, rcond=None)[0].T
        np.testing.assert_allclose(st.A, A, rtol=1e-9, atol=1e-11)
        np.testing.assert_allclose(st.B, B, rtol=1e-9, atol=1e-11)


# ------------------------------------------- step-size safeguard (reading of Sec. 7, App. B)
def _guard_case():
    m, n, r = 240, 200, 8
    row_ptr, col, val = gen.random_sparse(m, n, 0.1, 6)
    S = salsa.csr_matrix(m, n, row_ptr, col, val)
    W, H = gen.sign_constrained_init(m, n, r, float(val.mean()), 9)
    return S, W, H


def test_guard_without_rises_equals_plain_sweeps():
    """When no sweep raises the objective beyond the tolerance the safeguard is inert: the
    factors, momenta and counter equal those of plain sweeps exactly."""
    S, W, H = _guard_case()
    ST = S.T.tocsr()
    a = salsa.State(W, H)
    eta, fs, rej = salsa.guarded_sweeps(S, ST, a, 60, 50, 3, 3, "stochastic", 0.3, 0.5,
                                        tol=0.5)
    b = salsa.State(W, H)
    for _ in range(3):
        salsa.sweep(S, ST, b, 60, 50, 3, "stochastic", 0.3, 0.5)
    assert rej == [] and eta == 0.3 and len(fs) == 4
    for x, y in ((a.A, b.A), (a.B, b.B), (a.VA, b.VA), (a.VB, b.VB)):
        assert np.array_equal(x, y)
    assert a.t == b.t == 3
    assert abs(fs[-1] - salsa.objective(S, b.W, b.H)) == 0.0


def test_guard_replays_as_plain_sweeps_with_restarts():
    """A diverging setting (eta = 1, momentum 0.9, 20-row blocks): the safeguard's result equals
    plain sweeps in which each rejected attempt is dropped, the momenta are cleared and the step
    size halved before the same sweep is repeated.  Each rejected attempt really raised the
    objective and each accepted one did not (the rule's invariant), and the block order of a
    repeated sweep is that of its counter."""
    S, W, H = _guard_case()
    ST = S.T.tocsr()
    g = salsa.State(W, H)
    eta_end, fs, rej = salsa.guarded_sweeps(S, ST, g, 20, 20, 3, 6, "stochastic", 1.0, 0.9)
    assert len(rej) >= 3
    st = salsa.State(W, H)
    eta, f_prev, log = 1.0, salsa.objective(S, W, H), list(rej)
    accepted = [f_prev]
    for t in range(6):
        while log and log[0][0] == t:
            t_rej, eta_rej, f_rej = log.pop(0)
            assert eta_rej == eta
            trial = salsa.State(st.W, st.H)
            trial.VA, trial.VB, trial.t = st.VA.copy(), st.VB.copy(), st.t
            salsa.sweep(S, ST, trial, 20, 20, 3, "stochastic", eta, 0.9)
            f_trial = salsa.objective(S, trial.W, trial.H)
            assert f_trial == f_rej and f_trial > f_prev
            st.VA[:] = 0.0
            st.VB[:] = 0.0
            eta *= 0.5
        assert st.t == t
        salsa.sweep(S, ST, st, 20, 20, 3, "stochastic", eta, 0.9)
        f = salsa.objective(S, st.W, st.H)
        assert f <= f_prev
        accepted.append(f)
        f_prev = f
    assert eta == eta_end and accepted == fs
    assert np.array_equal(st.A, g.A) and np.array_equal(st.B, g.B)
    with pytest.raises(ValueError):
        salsa.guarded_sweeps(S, ST, salsa.State(W, H), 20, 20, 3, 6, "stochastic", 1.0, 0.9,
                             eta_min=0.3)
