"""GPU parity: libnmd (HIP, gfx950) against the fp64 oracle on the same seeded fp32 inputs.

Bars:
  * the block schedule and the per-block nonzero counts: bit-exact (checked on the host side
    in test_abi_host.py, repeated here for the GPU workloads);
  * W, H after one sweep and the objective: relative Frobenius error <= 1e-4;
  * the standalone rectified contraction (one fp32 accumulation, no solve): <= 2e-5.
Every test prints the case it runs before touching the GPU.
"""

import itertools
import math

import numpy as np
import pytest
import torch

from oracle import partition, salsa, schedule
from workloads import gen

import paper_2608_21607_amd as nmd

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _say(*a):
    print("[case]", *a, flush=True)


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def make_ctx(p, mode=None, eta=None, mom=None, seed=None, flags=0):
    ctx = nmd.Context(p.m, p.n, p.r, p.block_m, p.block_n, seed=p.seed if seed is None else seed,
                      mode=p.mode if mode is None else mode, eta=p.eta if eta is None else eta,
                      momentum=p.momentum if mom is None else mom, flags=flags)
    ctx.set_sparse_csr(p.row_ptr, p.col, p.val)
    return ctx


def gpu_run(p, sweeps, W0=None, H0=None, **kw):
    ctx = make_ctx(p, **kw)
    W = dev(p.W0 if W0 is None else W0)
    H = dev(p.H0 if H0 is None else H0)
    ctx.sweep(W, H, sweeps)
    torch.cuda.synchronize()
    return W.cpu().numpy(), H.cpu().numpy(), ctx


def oracle_run(p, sweeps, W0=None, H0=None, mode=None, eta=None, mom=None, seed=None):
    S = salsa.csr_matrix(p.m, p.n, p.row_ptr, p.col, p.val)
    st = salsa.State(p.W0 if W0 is None else W0, p.H0 if H0 is None else H0)
    ST = S.T.tocsr()
    for _ in range(sweeps):
        salsa.sweep(S, ST, st, p.block_m, p.block_n, p.seed if seed is None else seed,
                    mode=p.mode if mode is None else mode, eta=p.eta if eta is None else eta,
                    gamma=p.momentum if mom is None else mom)
    return st.W, st.H, S


def oracle_run_counting(p, sweeps):
    """oracle_run in the context's stochastic mode, also counting the positive entries of
    L = X P_J^T (eq. rectify) met by every step, from the state before the step."""
    S = salsa.csr_matrix(p.m, p.n, p.row_ptr, p.col, p.val)
    ST = S.T.tocsr()
    st = salsa.State(p.W0, p.H0)
    rb, cb = partition.bounds(p.m, p.block_m), partition.bounds(p.n, p.block_n)
    npos = 0
    for t in range(sweeps):
        for code in schedule.sweep_schedule(p.seed, t, len(rb) - 1, len(cb) - 1, True):
            X, P = (st.A, st.B[cb[code - 1]:cb[code]]) if code > 0 else \
                   (st.B, st.A[rb[-code - 1]:rb[-code]])
            for r0 in range(0, X.shape[0], 4096):
                npos += int(np.count_nonzero(X[r0:r0 + 4096] @ P.T > 0))
            salsa.run_steps(S, ST, st, [code], p.block_m, p.block_n, p.eta, p.momentum)
        st.t += 1
    return st.W, st.H, S, npos


def test_gpu_is_gfx950():
    assert torch.cuda.is_available()
    name = torch.cuda.get_device_properties(0).gcnArchName
    assert name.startswith("gfx950"), name


# ------------------------------------------------------------------ the dense kernel alone
@pytest.mark.parametrize("r", [16, 32, 48, 64, 128, 192, 256, 320, 384, 448, 512])
def test_rectified_contraction_kernel(r):
    rows, blk = 333 + r % 7, 517
    _say("rectified_contraction", rows, blk, r)
    g = np.random.default_rng(r)
    A = g.standard_normal((rows, r)).astype(np.float32)
    B = g.standard_normal((blk, r)).astype(np.float32)
    Y = nmd.rectified_contraction(dev(A), dev(B))
    torch.cuda.synchronize()
    want = salsa.rectified_contraction(A, B)
    assert rel(Y.cpu().numpy(), want) < 2e-5


def _sparse_sign_case(rows, blk, r, seed):
    """A > 0 and B < 0 (S-hat = 0) except a few panel rows flipped positive, so that only some
    16-row panel blocks (and within them only some entries) have a positive L."""
    g = np.random.default_rng(seed)
    A = np.abs(g.standard_normal((rows, r))).astype(np.float32)
    B = -np.abs(g.standard_normal((blk, r))).astype(np.float32)
    flip = g.choice(blk, max(1, blk // 40), replace=False)
    B[flip] = g.standard_normal((flip.size, r)).astype(np.float32)
    return A, B


@pytest.mark.parametrize("r", [16, 48, 64, 256, 512])
def test_rectified_contraction_skips_zero_blocks(r):
    """Panel blocks without a positive L are skipped: the result still matches the oracle on a
    mostly-zero S-hat with a ragged panel tail, and an all-negative L gives exactly zero."""
    rows, blk = 300 + r % 5, 1000 + 9
    _say("rectified_contraction sparse S-hat", rows, blk, r)
    A, B = _sparse_sign_case(rows, blk, r, r + 1)
    Y = nmd.rectified_contraction(dev(A), dev(B))
    torch.cuda.synchronize()
    want = salsa.rectified_contraction(A, B)
    assert np.count_nonzero(want) > 0
    assert rel(Y.cpu().numpy(), want) < 2e-5
    Y0 = nmd.rectified_contraction(dev(A), dev(-np.abs(B)))
    torch.cuda.synchronize()
    assert not torch.any(Y0 != 0).item()


def _thin_positive_case(rows, blk, r, seed, terms=8, p=0.06):
    """A > 0 and B < 0, plus `terms` rank-one terms u v^T with sparse random supports in the
    last columns: L is positive only where some term has both its row and its panel row, so
    most 16 x 4 slices of max(0, L) hold 0 to 4 positive entries at scattered positions."""
    g = np.random.default_rng(seed)
    A = np.abs(g.standard_normal((rows, r))).astype(np.float32)
    B = -np.abs(g.standard_normal((blk, r))).astype(np.float32)
    big = np.float32(2.0 * np.sqrt(r))
    for t in range(terms):
        c = r - 1 - t
        A[:, c] = np.where(g.random(rows) < p, big, 0.0)
        B[:, c] = np.where(g.random(blk) < p, big, 0.0)
    return A, B


@pytest.mark.parametrize("r", [128, 256, 512])
def test_rectified_contraction_thin_slices(r):
    """Scattered positive entries of max(0, L) (few per 16 x 4 slice, the regime of the
    sweeps): matches the oracle, with ragged row and panel counts."""
    rows, blk = 300 + r % 7, 1000 + 9
    _say("rectified_contraction thin slices", rows, blk, r)
    A, B = _thin_positive_case(rows, blk, r, 7 * r + 1)
    want = salsa.rectified_contraction(A, B)
    L = A.astype(np.float64) @ B.astype(np.float64).T
    density = float(np.mean(L > 0))
    assert 0.002 < density < 0.05, density
    Y = nmd.rectified_contraction(dev(A), dev(B))
    torch.cuda.synchronize()
    assert rel(Y.cpu().numpy(), want) < 2e-5


@pytest.mark.parametrize("r", [16, 32, 64, 128])
def test_rectified_contraction_paper_shape_sampled(r):
    """The kernel at the shape of the paper's throughput table (A: 250000 x r, B: 2500 x r);
    64 sampled output rows against the oracle."""
    rows, blk = 250_000, 2500
    _say("rectified_contraction paper shape", rows, blk, r)
    g = torch.Generator(device="cuda").manual_seed(r)
    A = torch.randn((rows, r), generator=g, device="cuda")
    B = torch.randn((blk, r), generator=g, device="cuda")
    Y = nmd.rectified_contraction(A, B)
    torch.cuda.synchronize()
    idx = np.random.default_rng(r).choice(rows, 64, replace=False)
    want = salsa.rectified_contraction(A[idx].cpu().numpy(), B.cpu().numpy())
    assert rel(Y[idx].cpu().numpy(), want) < 2e-5


@pytest.mark.parametrize("split", [False, True])
@pytest.mark.parametrize("rows,blk", [(500_000, 7142), (50_000, 16130)])
def test_rectified_contraction_cooccurrence_shapes_sampled(rows, blk, split):
    """r = 512 at the co-occurrence workload's step shapes (W-step: 500000 rows against a 7142-row
    panel; H-step: 50000 rows against 16130), N(0,1) factors so that every tile runs the second
    product; 64 sampled output rows against the oracle, fp32 and split bf16."""
    r = 512
    _say("rectified_contraction co-occurrence shape", rows, blk, r, "split" if split else "fp32")
    g = torch.Generator(device="cuda").manual_seed(rows + blk)
    A = torch.randn((rows, r), generator=g, device="cuda")
    B = torch.randn((blk, r), generator=g, device="cuda")
    Y = nmd.rectified_contraction_bf16x3(A, B) if split else nmd.rectified_contraction(A, B)
    torch.cuda.synchronize()
    idx = np.random.default_rng(rows + blk).choice(rows, 64, replace=False)
    want = salsa.rectified_contraction(A[idx].cpu().numpy(), B.cpu().numpy())
    e = rel(Y[idx].cpu().numpy(), want)
    print(f"r = 512 at {rows} x {blk} ({'split' if split else 'fp32'}): rel err {e:.2e}")
    assert e < (SPLIT_TOL if split else 2e-5)
    del A, B, Y


def test_graph_tenth_two_sweeps_quad_column_second_product():
    """The graph workload at a tenth of its size (13926 x 13926, r = 256, ~1.7M nonzeros), two
    stochastic sweeps.  Sweep 0 starts with S-hat = 0; in sweep 1 S-hat is sparse and positive,
    and the dense kernel's second product runs per quad-column (4 rows x 1 panel row) holding
    a positive entry (the counters show it).  W, H and the objective against the oracle."""
    p = gen.config(4, scale=0.1)
    _say("graph workload at scale 0.1, two sweeps", p.m, p.n, p.nnz)
    ctx = make_ctx(p)
    W, H = dev(p.W0), dev(p.H0)
    ctx.sweep(W, H, 1)
    ctx.dense_blocks(reset=True)
    ctx.sweep(W, H, 1)
    run, total, entries = ctx.dense_blocks()
    print(f"second sweep: {run} of {total} slices run whole, {entries} positive entries")
    assert total > 0 and 0 <= run <= total and entries > 0
    assert ctx.dense_blocks(reset=True) == (run, total, entries)
    assert ctx.dense_blocks() == (0, 0, 0)
    Wg, Hg = W.cpu().numpy(), H.cpu().numpy()
    Wo, Ho, S = oracle_run(p, 2)
    ew, eh = rel(Wg, Wo), rel(Hg, Ho)
    print(f"two sweeps: rel err W {ew:.2e} H {eh:.2e}")
    assert ew < TOL and eh < TOL
    f = ctx.objective(W, H)
    assert abs(f - salsa.objective(S, Wg, Hg)) <= TOL * f


def test_graph_tenth_block_grid_17x17_two_sweeps():
    """The graph workload at a tenth of its size with the full workload's block grid: 13926 x
    13926 split into 17 x 17 blocks of 819-820 rows and columns (r = 256, the workload's step
    size and momentum), two stochastic sweeps of 34 steps each, end to end.  W, H and the
    objective against the oracle."""
    p = gen.config(4, scale=0.1)
    p.block_m = p.block_n = -(-p.m // 17)
    assert partition.num_blocks(p.m, p.block_m) == 17
    _say("graph workload at scale 0.1, 17 x 17 blocks, two sweeps", p.m, p.nnz, p.block_m)
    ctx = make_ctx(p)
    W, H = dev(p.W0), dev(p.H0)
    ctx.sweep(W, H, 2)
    Wg, Hg = W.cpu().numpy(), H.cpu().numpy()
    Wo, Ho, S = oracle_run(p, 2)
    ew, eh = rel(Wg, Wo), rel(Hg, Ho)
    f_gpu, f_orc = ctx.objective(W, H), salsa.objective(S, Wo, Ho)
    print(f"17 x 17 blocks, two sweeps: rel err W {ew:.2e} H {eh:.2e}; f gpu {f_gpu:.6f} "
          f"oracle {f_orc:.6f} (start {salsa.objective(S, p.W0, p.H0):.6f})")
    assert ew < TOL and eh < TOL
    assert abs(f_gpu - f_orc) <= TOL * f_orc


# ---------------------------------------------- split-bf16 products (both products, bf16x3)
# Each product carries a relative error of about 2^-16 of the sum of the magnitudes of its terms
# (three bf16 products of two-term splits).  Against the fp64 oracle that is of order 1e-5 on Y
# for N(0,1) factors.
SPLIT_TOL = 1e-4


@pytest.mark.parametrize("r,rows,blk", [(16, 700, 999), (32, 300, 1000), (64, 257, 517), (128, 129, 33),
                                         (128, 1000, 2500), (256, 340, 517), (64, 5, 7),
                                         (512, 300, 517), (512, 70, 31), (512, 129, 96),
                                         (256, 5, 7), (256, 1, 1), (512, 1, 1), (512, 17, 33)])
def test_rectified_contraction_bf16x3(r, rows, blk):
    """Both products on split bf16: N(0,1) factors (about half of L positive, every 16 x 32
    tile live), ragged rows and panel sizes (a panel shorter than one 32-row pair included)."""
    _say("rectified_contraction_bf16x3", rows, blk, r)
    g = np.random.default_rng(1000 * r + blk)
    A = g.standard_normal((rows, r)).astype(np.float32)
    B = g.standard_normal((blk, r)).astype(np.float32)
    Y = nmd.rectified_contraction_bf16x3(dev(A), dev(B))
    torch.cuda.synchronize()
    e = rel(Y.cpu().numpy(), salsa.rectified_contraction(A, B))
    print(f"bf16x3 r = {r}: rel err {e:.2e}")
    assert e < SPLIT_TOL


@pytest.mark.parametrize("r", [16, 32, 128, 256, 512])
def test_rectified_contraction_bf16x3_sparse_and_zero(r):
    """Thin positive slices (most 16 x 32 tiles skipped) and an all-negative L (exact zero)."""
    rows, blk = 300 + 4, 1000 + 9
    _say("rectified_contraction_bf16x3 sparse", rows, blk, r)
    A, B = _thin_positive_case(rows, blk, r, 11 * r + 3)
    Y = nmd.rectified_contraction_bf16x3(dev(A), dev(B))
    torch.cuda.synchronize()
    e = rel(Y.cpu().numpy(), salsa.rectified_contraction(A, B))
    print(f"bf16x3 thin slices r = {r}: rel err {e:.2e}")
    assert e < SPLIT_TOL
    Y0 = nmd.rectified_contraction_bf16x3(dev(np.abs(A)), dev(-np.abs(B)))
    torch.cuda.synchronize()
    assert not torch.any(Y0 != 0).item()


@pytest.mark.parametrize("r", [64, 256, 512])
def test_rectified_contraction_bf16x3_workspace_reuse(r):
    """Two calls in a row on one workspace, the second with a shorter panel: the second result
    depends only on its own inputs."""
    _say("rectified_contraction_bf16x3 workspace reuse", 200, 700, r)
    g = np.random.default_rng(77 + r)
    A = g.standard_normal((200, r)).astype(np.float32)
    B1 = g.standard_normal((700, r)).astype(np.float32)
    B2 = g.standard_normal((45, r)).astype(np.float32)
    work = torch.empty((nmd.bf16x3_workspace_floats(700, r),), device="cuda")
    nmd.rectified_contraction_bf16x3(dev(A), dev(B1), work=work)
    Y = nmd.rectified_contraction_bf16x3(dev(A), dev(B2), work=work)
    torch.cuda.synchronize()
    assert rel(Y.cpu().numpy(), salsa.rectified_contraction(A, B2)) < SPLIT_TOL


def test_graph_tenth_two_sweeps_split_bf16():
    """The graph workload at a tenth of its size, two stochastic sweeps with both products of the
    dense term on split bf16: W, H and the objective within the 1e-4 bar of the fp64 oracle."""
    p = gen.config(4, scale=0.1)
    _say("graph workload at scale 0.1, two sweeps, split bf16", p.m, p.n, p.nnz)
    ctx = make_ctx(p, flags=nmd.FLAG_SPLIT_BF16)
    W, H = dev(p.W0), dev(p.H0)
    ctx.sweep(W, H, 2)
    run, total, entries = ctx.dense_blocks()
    # the both-products kernel counts its live 16 x 32 tiles as 8 slices each, and (r_p = 256)
    # the positive entries of max(0, L) it met, which the oracle counts on its own trajectory
    assert total > 0 and run > 0 and run % 8 == 0
    Wg, Hg = W.cpu().numpy(), H.cpu().numpy()
    Wo, Ho, S, npos = oracle_run_counting(p, 2)
    print(f"positive entries of max(0, L): gpu {entries}, oracle {npos}")
    assert abs(entries - npos) <= 1e-3 * npos + 16
    ew, eh = rel(Wg, Wo), rel(Hg, Ho)
    print(f"split bf16, two sweeps: rel err W {ew:.2e} H {eh:.2e}")
    assert ew < TOL and eh < TOL
    f = ctx.objective(W, H)
    assert abs(f - salsa.objective(S, Wg, Hg)) <= TOL * f


# -------------------------------------------------------------- whole sweeps, small problems
def test_config1_deterministic_three_sweeps():
    p = gen.config(1)
    _say("config 1 deterministic, 3 sweeps")
    Wg, Hg, ctx = gpu_run(p, 1)
    Wo, Ho, S = oracle_run(p, 1)
    assert rel(Wg, Wo) < TOL and rel(Hg, Ho) < TOL
    Wg3, Hg3, ctx3 = gpu_run(p, 3)
    Wo3, Ho3, _ = oracle_run(p, 3)
    assert rel(Wg3, Wo3) < 3 * TOL and rel(Hg3, Ho3) < 3 * TOL
    f_gpu = ctx3.objective(dev(Wg3), dev(Hg3))
    f_orc = salsa.objective(S, Wg3, Hg3)
    assert abs(f_gpu - f_orc) <= TOL * f_orc
    f0 = ctx3.objective(dev(p.W0), dev(p.H0))
    assert abs(f0 - salsa.objective(S, p.W0, p.H0)) <= TOL * f0
    assert f_gpu < f0
    assert ctx3.sweep_count == 3


def test_deterministic_objective_monotone_on_gpu():
    p = gen.config(1)
    _say("config 1 monotone over 6 sweeps")
    ctx = make_ctx(p)
    W, H = dev(p.W0), dev(p.H0)
    f = ctx.objective(W, H)
    for _ in range(6):
        ctx.sweep(W, H, 1)
        f1 = ctx.objective(W, H)
        assert f1 <= f * (1 + 1e-5)
        f = f1


def fp32_objective_bound(S, W, H):
    """|f(L_fp32) - f(L)| <= ||L_fp32 - L||_F / ||S||_F because f is a distance to a closed
    convex set (1-Lipschitz); each entry of an fp32 dot product of length r errs by at most
    gamma_r sum_k |w_ik h_kj|, gamma_r = r u / (1 - r u), u = 2^-24, in any summation order."""
    r = W.shape[1]
    u = 2.0 ** -24
    gamma = r * u / (1 - r * u)
    absL = np.abs(np.asarray(W, np.float64)) @ np.abs(np.asarray(H, np.float64))
    return gamma * np.linalg.norm(absL) / math.sqrt(float(S.multiply(S).sum()))


@pytest.mark.parametrize("n", [256, 4096])
def test_identity_exact_completion(n):
    """Corollary 1: the rank-3 completion of I_n is an exact fixed point.  In fp32 its
    objective is not zero (entries of size n^2/pi^2 cancel), so the GPU objective is compared
    with the oracle's objective at the same fp32-rounded factors, within the fp32 dot-product
    error bound."""
    _say("identity exact factors", n)
    W, H = gen.identity_exact_factors(n, np.float32)
    row_ptr, col, val = gen.identity(n)
    p = gen.Problem("identity", n, n, 3, row_ptr, col, val, W, H, min(1024, n), min(1024, n))
    Wg, Hg, ctx = gpu_run(p, 1)
    Wo, Ho, S = oracle_run(p, 1)
    assert rel(Wg, Wo) < TOL and rel(Hg, Ho) < TOL
    assert rel(Wg, W) < 1e-3 and rel(Hg, H) < 1e-3  # stays at the fixed point
    f_gpu = ctx.objective(dev(W), dev(H))
    f_orc = salsa.objective(S, W, H)
    bound = fp32_objective_bound(S, W, H)
    print(f"identity n={n}: f_gpu={f_gpu:.3e} f_orc={f_orc:.3e} bound={bound:.3e}")
    assert f_orc < 0.1
    assert abs(f_gpu - f_orc) <= bound


def test_config2_identity_random_init():
    p = gen.config(2)
    _say("config 2 identity, random init, 1 sweep")
    Wg, Hg, ctx = gpu_run(p, 1)
    Wo, Ho, S = oracle_run(p, 1)
    assert rel(Wg, Wo) < TOL and rel(Hg, Ho) < TOL
    f_gpu = ctx.objective(dev(Wg), dev(Hg))
    assert abs(f_gpu - salsa.objective(S, Wg, Hg)) <= TOL * f_gpu


@pytest.mark.parametrize("eta,mom", [(1.0, 0.0), (1.0, 0.9), (0.5, 0.0), (0.5, 0.9)])
def test_stochastic_planted_reduced(eta, mom):
    p = gen.config(3, scale=0.125)  # 4096 x 4096, r = 64
    p.block_m = p.block_n = 512
    _say("config 3 reduced, stochastic", eta, mom)
    Wg, Hg, ctx = gpu_run(p, 1, eta=eta, mom=mom)
    Wo, Ho, S = oracle_run(p, 1, eta=eta, mom=mom)
    assert rel(Wg, Wo) < TOL and rel(Hg, Ho) < TOL
    R, C = partition.num_blocks(p.m, 512), partition.num_blocks(p.n, 512)
    assert ctx.schedule(0) == schedule.sweep_schedule(p.seed, 0, R, C, True)


@pytest.mark.parametrize("case", ["r64_fused", "r128_multi", "r320_fused"])
def test_long_runs_of_same_side_steps(case):
    """Uneven block grids, so that the schedule has runs of more than eight H-steps (21 or 20
    row blocks against 2 or 1 column blocks): their solves are formed in batches of up to
    eight, by the single-workgroup form at r_p = 64 and 320 and the multi-launch form at 128.
    One sweep, momentum 0.9, against the oracle."""
    if case == "r320_fused":
        p = gen.config(4, scale=0.1)  # 13926 x 13926 graph-like counts
        r, p.block_m, p.block_n = 320, 700, p.n
    else:
        p = gen.config(3, scale=0.125)  # 4096 x 4096 planted
        r, p.block_m, p.block_n = (64 if case == "r64_fused" else 128), 200, 2048
    if r != p.r:
        p.r = r
        p.W0, p.H0 = gen.sign_constrained_init(p.m, p.n, r, float(p.val.mean()), 1003)
    R, C = partition.num_blocks(p.m, p.block_m), partition.num_blocks(p.n, p.block_n)
    codes = schedule.sweep_schedule(p.seed, 0, R, C, True)
    assert max(sum(1 for _ in g) for _, g in itertools.groupby(codes, key=lambda c: c > 0)) > 8
    _say("long runs of same-side steps", case, p.m, p.n, r, R, C)
    Wg, Hg, _ = gpu_run(p, 1, mode="stochastic", eta=1.0, mom=0.9)
    Wg2, Hg2, _ = gpu_run(p, 1, mode="stochastic", eta=1.0, mom=0.9)
    assert np.array_equal(Wg, Wg2) and np.array_equal(Hg, Hg2)  # batched solves deterministic
    Wo, Ho, _ = oracle_run(p, 1, mode="stochastic", eta=1.0, mom=0.9)
    ew, eh = rel(Wg, Wo), rel(Hg, Ho)
    print(f"{case}: rel err W {ew:.2e} H {eh:.2e}")
    assert ew < TOL and eh < TOL


def test_stochastic_planted_reduced_split_bf16():
    """The split-bf16 flag at r_p = 64 (the 32 x 32 x 16 form of both products) on the 4096 x 4096
    planted workload, momentum 0.9, one sweep: W, H within the 1e-4 bar."""
    p = gen.config(3, scale=0.125)
    p.block_m = p.block_n = 512
    _say("config 3 reduced, stochastic, split bf16")
    ctx = make_ctx(p, eta=1.0, mom=0.9, flags=nmd.FLAG_SPLIT_BF16)
    W, H = dev(p.W0), dev(p.H0)
    ctx.sweep(W, H, 1)
    run, total, entries = ctx.dense_blocks()
    assert total > 0 and run % 16 == 0 and entries == 0  # live 32 x 32 tiles count 16 slices
    Wo, Ho, _ = oracle_run(p, 1, eta=1.0, mom=0.9)
    ew, eh = rel(W.cpu().numpy(), Wo), rel(H.cpu().numpy(), Ho)
    print(f"split bf16 sweep r = 64: rel err W {ew:.2e} H {eh:.2e}")
    assert ew < TOL and eh < TOL


@pytest.mark.parametrize("r", [200, 480])
def test_graph_small_split_bf16_padded_rank(r):
    """The split-bf16 flag at ranks that pad (200 -> 256, 480 -> 512: the staged kernels with
    zero padding columns) on the graph workload at a tenth of its size (two 8192-row blocks per
    side), two stochastic sweeps, so that the second product runs in the second: W, H within
    the 1e-4 bar.  (Much smaller problems at these ranks amplify any perturbation several-fold
    per sweep, fp32 included, or leave the oracle's Gram matrices singular.)"""
    p = gen.config(4, scale=0.1)
    p.r = r
    p.W0, p.H0 = gen.sign_constrained_init(p.m, p.n, r, float(p.val.mean()), 1004)
    _say("graph workload at scale 0.1, split bf16, padded rank", p.m, p.n, r)
    ctx = make_ctx(p, flags=nmd.FLAG_SPLIT_BF16)
    W, H = dev(p.W0), dev(p.H0)
    ctx.sweep(W, H, 2)
    run, total, entries = ctx.dense_blocks()
    assert total > 0 and run > 0 and entries > 0  # entries: positive entries of max(0, L)
    Wo, Ho, _ = oracle_run(p, 2)
    ew, eh = rel(W.cpu().numpy(), Wo), rel(H.cpu().numpy(), Ho)
    print(f"split bf16, r = {r}, two sweeps: rel err W {ew:.2e} H {eh:.2e}, live slices {run / total:.3f}")
    assert ew < TOL and eh < TOL


def test_stochastic_three_sweeps_and_persistent_state():
    """Sweeps run in one call equal the same sweeps run one call at a time (the sweep counter
    and the momentum persist); after reset the first sweep repeats bit for bit."""
    p = gen.config(3, scale=0.0625)
    p.block_m = p.block_n = 512
    _say("persistent state", p.m, p.n)
    W1, H1, _ = gpu_run(p, 3)
    ctx = make_ctx(p)
    W, H = dev(p.W0), dev(p.H0)
    for _ in range(3):
        ctx.sweep(W, H, 1)
    assert np.array_equal(W.cpu().numpy(), W1) and np.array_equal(H.cpu().numpy(), H1)
    Wo, Ho, _ = oracle_run(p, 3)
    assert rel(W1, Wo) < 3 * TOL and rel(H1, Ho) < 3 * TOL
    ctx.reset()
    W, H = dev(p.W0), dev(p.H0)
    ctx.sweep(W, H, 1)
    Wa, Ha, _ = gpu_run(p, 1)
    assert np.array_equal(W.cpu().numpy(), Wa) and np.array_equal(H.cpu().numpy(), Ha)


ODD = [
    # m, n, r, block_m, block_n, mode, eta, mom, extras
    (37, 53, 1, 10, 13, "stochastic", 1.0, 0.0, {}),
    (100, 77, 3, 33, 20, "stochastic", 0.5, 0.9, {"empty_rows": 3, "empty_cols": 2}),
    (129, 300, 8, 64, 100, "deterministic", 1.0, 0.0, {"heavy_row_frac": 0.5}),
    (257, 65, 17, 100, 33, "stochastic", 1.0, 0.9, {}),
    (300, 410, 64, 150, 205, "stochastic", 1.0, 0.9, {"heavy_row_frac": 0.5}),
    (333, 290, 100, 333, 290, "deterministic", 1.0, 0.0, {"empty_rows": 5}),
    (700, 600, 256, 350, 300, "stochastic", 1.0, 0.9, {}),
    (1100, 900, 512, 550, 900, "stochastic", 1.0, 0.0, {"heavy_row_frac": 0.3}),
    # deterministic at r_p = 320: the correction beside the dense kernel, a W-step's two column
    # blocks written and then added into its buffer
    (600, 500, 320, 200, 250, "deterministic", 1.0, 0.0, {"heavy_row_frac": 0.3}),
]


@pytest.mark.parametrize("case", ODD, ids=[f"{c[0]}x{c[1]}r{c[2]}" for c in ODD])
def test_odd_shapes(case):
    m, n, r, bm, bn, mode, eta, mom, extras = case
    _say("odd shape", case)
    row_ptr, col, val = gen.random_sparse(m, n, 0.05, m + n + r, **extras)
    W0, H0 = gen.sign_constrained_init(m, n, r, float(val.mean()), r)
    p = gen.Problem("odd", m, n, r, row_ptr, col, val, W0, H0, bm, bn, mode, eta, mom, 7)
    Wg, Hg, ctx = gpu_run(p, 1)
    Wo, Ho, S = oracle_run(p, 1)
    assert rel(Wg, Wo) < TOL and rel(Hg, Ho) < TOL
    f = ctx.objective(dev(Wg), dev(Hg))
    assert abs(f - salsa.objective(S, Wg, Hg)) <= TOL * f


# Stochastic sweeps on nearly full and 26% full matrices at the quad-column ranks: many nonzeros
# on every row of every block, for the sparse correction's long rows (items cut into several
# parts) and the second product's dense slices.  (At r = 512 the blocks keep 700 panel rows:
# with 550 the Gram matrices of a nearly full S are conditioned badly enough that fp32 rounding
# alone moves W and H by 2e-4 from the fp64 oracle.)
DENSE_ROWS = [(700, 600, 256, 350, 300, 3.0), (700, 600, 256, 350, 300, 0.3),
              (1400, 1400, 512, 700, 700, 3.0)]


@pytest.mark.parametrize("case", DENSE_ROWS,
                         ids=[f"{c[0]}x{c[1]}r{c[2]}d{c[5]}" for c in DENSE_ROWS])
def test_dense_rows_sweep(case):
    m, n, r, bm, bn, density = case
    _say("dense rows, one stochastic sweep", case)
    row_ptr, col, val = gen.random_sparse(m, n, density, m + n + r + 11)
    W0, H0 = gen.sign_constrained_init(m, n, r, float(val.mean()), r + 1)
    p = gen.Problem("dense rows", m, n, r, row_ptr, col, val, W0, H0, bm, bn, "stochastic", 1.0,
                    0.9, 7)
    Wg, Hg, ctx = gpu_run(p, 1)
    Wo, Ho, S = oracle_run(p, 1)
    ew, eh = rel(Wg, Wo), rel(Hg, Ho)
    print(f"nnz {len(col)}: rel err W {ew:.2e} H {eh:.2e}")
    assert ew < TOL and eh < TOL
    f = ctx.objective(dev(Wg), dev(Hg))
    assert abs(f - salsa.objective(S, Wg, Hg)) <= TOL * f


# ---------------------------------------------------------- objective and reconstruction metrics
def test_metrics_calibration_and_fit():
    """eqs. RMSE and WJD: at the sign-constrained start S-hat = 0, so both equal 1 (their
    calibration); after three deterministic sweeps all three measures match the oracle
    at the same factors, and the objective bounds the RMSE from above (Prop. 9)."""
    p = gen.config(1)
    _say("metrics, config 1")
    ctx = make_ctx(p)
    S = salsa.csr_matrix(p.m, p.n, p.row_ptr, p.col, p.val)
    m0 = ctx.metrics(dev(p.W0), dev(p.H0))
    # ||S||_F summed on the device over the host's ||S||_F: equal up to fp64 summation order
    assert abs(m0["rmse"] - 1.0) <= 1e-12 and m0["wjd"] == 1.0
    assert abs(m0["objective"] - ctx.objective(dev(p.W0), dev(p.H0))) <= 1e-12
    W, H = dev(p.W0), dev(p.H0)
    ctx.sweep(W, H, 3)
    Wg, Hg = W.cpu().numpy(), H.cpu().numpy()
    m3 = ctx.metrics(W, H)
    assert abs(m3["objective"] - salsa.objective(S, Wg, Hg)) <= TOL * m3["objective"]
    assert abs(m3["rmse"] - salsa.rmse(S, Wg, Hg)) <= TOL * m3["rmse"]
    assert abs(m3["wjd"] - salsa.wjd(S, Wg, Hg)) <= TOL * m3["wjd"]
    assert m3["objective"] >= m3["rmse"] and m3["rmse"] < 1.0 and m3["wjd"] < 1.0
    assert abs(m3["objective"] - ctx.objective(W, H)) <= 1e-12 * m3["objective"]


@pytest.mark.parametrize("case", [(300, 410, 64), (333, 290, 100), (700, 600, 256), (600, 900, 512)],
                         ids=lambda c: f"{c[0]}x{c[1]}r{c[2]}")
def test_metrics_random_factors(case):
    """All three measures at random Gaussian factors (S-hat about half positive), every padded
    rank path of the objective kernel, against the oracle."""
    m, n, r = case
    _say("metrics, random factors", case)
    row_ptr, col, val = gen.random_sparse(m, n, 0.05, m + n + r, heavy_row_frac=0.3)
    g = np.random.default_rng(r)
    W0 = (g.standard_normal((m, r)) / math.sqrt(r)).astype(np.float32)
    H0 = g.standard_normal((r, n)).astype(np.float32)
    p = gen.Problem("metrics", m, n, r, row_ptr, col, val, W0, H0, 128, 128, "deterministic",
                    1.0, 0.0, 7)
    ctx = make_ctx(p)
    S = salsa.csr_matrix(m, n, row_ptr, col, val)
    got = ctx.metrics(dev(W0), dev(H0))
    assert abs(got["objective"] - salsa.objective(S, W0, H0)) <= TOL * got["objective"]
    assert abs(got["rmse"] - salsa.rmse(S, W0, H0)) <= TOL * got["rmse"]
    assert abs(got["wjd"] - salsa.wjd(S, W0, H0)) <= TOL * got["wjd"]
    assert got["objective"] >= got["rmse"]


def test_bitwise_determinism():
    p = gen.config(3, scale=0.0625)
    p.block_m = p.block_n = 256
    _say("determinism")
    W1, H1, _ = gpu_run(p, 2)
    W2, H2, _ = gpu_run(p, 2)
    assert np.array_equal(W1, W2) and np.array_equal(H1, H2)


# ------------------------------------------------------------------------------ error paths
def test_nonfinite_input_is_reported():
    p = gen.config(1)
    p.mode = "stochastic"
    _say("NaN in W")
    W0 = p.W0.copy()
    W0[5, 2] = np.nan
    ctx = make_ctx(p)
    W, H = dev(W0), dev(p.H0)
    with pytest.raises(nmd.NmdError) as e:
        ctx.sweep(W, H, 1)
    assert e.value.code == -6 and "sweep 0" in e.value.message


def test_singular_gram_is_reported_and_later_steps_skipped():
    p = gen.config(1)
    p.mode = "stochastic"
    _say("zero column block of H")
    H0 = p.H0.copy()
    first = gen_first_w_block(p)
    H0[:, first[0]:first[1]] = 0.0  # the first W-step's Gram matrix is zero
    ctx = make_ctx(p)
    W, H = dev(p.W0), dev(H0)
    with pytest.raises(nmd.NmdError) as e:
        ctx.sweep(W, H, 1)
    assert e.value.code == -4 and "step 0" in e.value.message
    assert np.array_equal(W.cpu().numpy(), p.W0)
    assert np.array_equal(H.cpu().numpy(), H0)


def test_rejected_step_keeps_last_completed_step():
    """A NaN in H outside the first W-step's column block: step 0 (that W-step) completes, the
    H-step after it carries the NaN into its output and is rejected.  W must come back exactly
    as after step 0 alone and H as given (the rejected step and the skipped ones leave the
    factors and momenta of the last completed step); after nmd_reset the context runs again."""
    p = gen.config(1)
    _say("NaN in H, rejected at step 1")
    first = gen_first_w_block(p)
    col = first[1] % p.n if first[1] < p.n else 0  # a column outside the first W block
    assert not (first[0] <= col < first[1])
    H0 = p.H0.copy()
    H0[3, col] = np.nan
    R, C = partition.num_blocks(p.m, p.block_m), partition.num_blocks(p.n, p.block_n)
    steps = schedule.sweep_schedule(p.seed, 0, R, C, True)[:3]
    assert steps[0] > 0 and steps[1] < 0
    kw = dict(mode="stochastic", eta=1.0, mom=0.9)
    ref = make_ctx(p, **kw)
    Wr, Hr = dev(p.W0), dev(H0)
    ref.run_steps(Wr, Hr, steps[:1])
    ctx = make_ctx(p, **kw)
    W, H = dev(p.W0), dev(H0)
    with pytest.raises(nmd.NmdError) as e:
        ctx.run_steps(W, H, steps)
    assert e.value.code == -6 and "step 1" in e.value.message
    assert np.array_equal(W.cpu().numpy(), Wr.cpu().numpy())
    assert np.array_equal(H.cpu().numpy(), H0, equal_nan=True)
    # after nmd_reset the context runs the same steps exactly as the reference does
    ctx.reset()
    ref.reset()
    W2, H2 = dev(p.W0), dev(p.H0)
    W3, H3 = dev(p.W0), dev(p.H0)
    ctx.run_steps(W2, H2, steps)
    ref.run_steps(W3, H3, steps)
    assert np.array_equal(W2.cpu().numpy(), W3.cpu().numpy())
    assert np.array_equal(H2.cpu().numpy(), H3.cpu().numpy())


@pytest.mark.parametrize("codes,bad,first_fail", [
    ((1, 2, 3), (3,), 2),       # the last step of a run of three W-steps
    ((1, 3, 2, 4), (3,), 1),    # a step inside a run: the one before it is kept
    ((3, 1, 4), (3, 4), 0),     # two singular steps in one run: the first is reported
    ((-1, -3, -2), (-3,), 1),   # the same on the H side (a zero row block of W)
])
def test_singular_gram_inside_a_run_of_steps(codes, bad, first_fail):
    """Consecutive steps of one side have their Gram matrices and solves formed together,
    ahead of their updates.  A step whose Gram matrix is singular stops itself and every later
    step, but the steps before it in the same run are kept: W and H come back exactly as after
    those steps alone."""
    p = gen.config(1)
    _say("singular Gram inside a run", codes, bad)
    bn, bm = partition.bounds(p.n, p.block_n), partition.bounds(p.m, p.block_m)
    W0, H0 = p.W0.copy(), p.H0.copy()
    for k in bad:
        if k > 0:
            H0[:, bn[k - 1]:bn[k]] = 0.0  # W-steps on column block k see a zero panel
        else:
            W0[bm[-k - 1]:bm[-k], :] = 0.0  # H-steps on row block -k see a zero panel
    kw = dict(mode="stochastic", eta=1.0, mom=0.9)
    ref = make_ctx(p, **kw)
    Wr, Hr = dev(W0), dev(H0)
    if first_fail:
        ref.run_steps(Wr, Hr, list(codes[:first_fail]))
    ctx = make_ctx(p, **kw)
    W, H = dev(W0), dev(H0)
    with pytest.raises(nmd.NmdError) as e:
        ctx.run_steps(W, H, list(codes))
    assert e.value.code == -4 and f"step {first_fail};" in e.value.message
    assert np.array_equal(W.cpu().numpy(), Wr.cpu().numpy())
    assert np.array_equal(H.cpu().numpy(), Hr.cpu().numpy())


def _solve_batches(codes, batch=8):
    """Runs of consecutive same-side steps, cut into pieces of at most `batch` steps."""
    n, i = 0, 0
    while i < len(codes):
        j = i
        while j < len(codes) and j - i < batch and (codes[j] > 0) == (codes[i] > 0):
            j += 1
        n, i = n + 1, j
    return n


def test_kernel_timing_counts_steps_and_runs():
    """With timing on, one sweep records a dense, sparse, update and join entry per step and one
    Gram-and-inverse entry per run of consecutive same-side steps (at most eight)."""
    p = gen.config(1)
    p.block_m, p.block_n = 64, 500  # 16 row blocks, 2 column blocks: runs of H-steps
    _say("kernel timing classes, 1000 x 1000 with 16 x 2 blocks")
    ctx = make_ctx(p, mode="stochastic", flags=nmd.FLAG_TIMING)
    W, H = dev(p.W0), dev(p.H0)
    ctx.sweep(W, H, 1)
    codes = list(ctx.schedule(0))
    assert len(codes) == 18
    t = [ctx.kernel_timing(k) for k in range(5)]
    for k in (0, 3, 4):
        assert t[k]["launches"] == len(codes), (k, t[k])
    assert t[1]["launches"] >= len(codes)  # one per block's share of the nonzeros
    assert t[2]["launches"] == _solve_batches(codes) < len(codes), (t[2], codes)
    assert t[0]["ms"] > 0 and t[2]["ms"] > 0 and t[4]["ms"] >= 0


def gen_first_w_block(p):
    R, C = partition.num_blocks(p.m, p.block_m), partition.num_blocks(p.n, p.block_n)
    code = schedule.sweep_schedule(p.seed, 0, R, C, True)[0]
    assert code > 0
    b = partition.bounds(p.n, p.block_n)
    return b[code - 1], b[code]


def test_bad_tensor_arguments():
    p = gen.config(1)
    ctx = make_ctx(p)
    with pytest.raises(ValueError):
        ctx.sweep(dev(p.W0.T), dev(p.H0), 1)
    with pytest.raises(TypeError):
        ctx.sweep(torch.from_numpy(p.W0), dev(p.H0), 1)
