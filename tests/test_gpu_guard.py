"""GPU: per-sweep objectives and the step-size safeguard against the oracle's rule.

The safeguard is a reading of Sec. 7 (stochastic updates diverge for too large a step size) and
of the appendix on experimental settings (the step size is lowered for the models that need
it): a sweep that raises the objective by more than a relative tolerance is undone, the momenta
are cleared, the step size is halved and the sweep is run again.  The library decides on the
device after each sweep; the oracle (salsa.guarded_sweeps) implements the same rule on its own.
The cases are chosen so that every decision has a margin far above the fp32 error, which the
test checks on the oracle side before comparing.
"""

import numpy as np
import pytest
import torch

from oracle import salsa
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


def _problem(m, n, r, density, seed):
    row_ptr, col, val = gen.random_sparse(m, n, density, seed)
    W0, H0 = gen.sign_constrained_init(m, n, r, float(val.mean()), 9)
    return row_ptr, col, val, W0, H0


def _ctx(m, n, r, blk, row_ptr, col, val, flags, eta=1.0, mom=0.9, tol=0.0, eta_min=0.0,
         mode="stochastic"):
    ctx = nmd.Context(m, n, r, blk, blk, seed=3, mode=mode, eta=eta, momentum=mom, flags=flags,
                      guard_tol=tol, eta_min=eta_min)
    ctx.set_sparse_csr(row_ptr, col, val)
    return ctx


def test_sweep_objectives_follow_the_trajectory():
    """NMD_FLAG_SWEEP_OBJECTIVE records f before and after every sweep (eq. auxCost) without
    changing the trajectory: W and H are bit-identical to a run without the flag, and each
    recorded f matches the oracle's objective after that sweep."""
    m, n, r, blk = 300, 260, 8, 64
    row_ptr, col, val, W0, H0 = _problem(m, n, r, 0.08, 2)
    _say("per-sweep objectives", m, n, r, blk)
    a = _ctx(m, n, r, blk, row_ptr, col, val, nmd.FLAG_SWEEP_OBJECTIVE, eta=0.5)
    b = _ctx(m, n, r, blk, row_ptr, col, val, 0, eta=0.5)
    Wa, Ha, Wb, Hb = dev(W0), dev(H0), dev(W0), dev(H0)
    a.sweep(Wa, Ha, 3)
    b.sweep(Wb, Hb, 3)
    assert np.array_equal(Wa.cpu().numpy(), Wb.cpu().numpy())
    assert np.array_equal(Ha.cpu().numpy(), Hb.cpu().numpy())
    f = a.sweep_objectives()
    assert f.shape == (4,)
    S = salsa.csr_matrix(m, n, row_ptr, col, val)
    st = salsa.State(W0, H0)
    fo = [salsa.objective(S, st.W, st.H)]
    for _ in range(3):
        salsa.sweep(S, S.T.tocsr(), st, blk, blk, 3, "stochastic", 0.5, 0.9)
        fo.append(salsa.objective(S, st.W, st.H))
    e = np.abs(f - fo) / np.asarray(fo)
    print("per-sweep f", np.round(f, 6), "max rel err", f"{e.max():.2e}")
    assert e.max() <= TOL
    assert rel(Wa.cpu().numpy(), st.W) <= TOL and rel(Ha.cpu().numpy(), st.H) <= TOL
    assert a.sweep_count == 3 and a.step_size() == (0.5, 0)
    # a second call records its own history, starting from the current factors
    a.sweep(Wa, Ha, 1)
    g = a.sweep_objectives()
    assert g.shape == (2,) and abs(g[0] - f[-1]) <= 1e-12 * f[-1]


@pytest.mark.parametrize("m,n,seed,tol", [(240, 200, 6, 0.0), (200, 150, 5, 0.01)])
def test_guard_matches_oracle_rule(m, n, seed, tol):
    """eta = 1, momentum 0.9 on 20-row blocks diverges within a sweep; the safeguard halves the
    step size several times.  The halvings, the accepted objectives and the final factors must
    match the oracle's implementation of the rule."""
    r, blk, sweeps = 8, 20, 8
    row_ptr, col, val, W0, H0 = _problem(m, n, r, 0.1, seed)
    S = salsa.csr_matrix(m, n, row_ptr, col, val)
    st = salsa.State(W0, H0)
    eta_o, fo, rej = salsa.guarded_sweeps(S, S.T.tocsr(), st, blk, blk, 3, sweeps, "stochastic",
                                          1.0, 0.9, tol=tol, eta_min=1e-3)
    # every decision of the oracle is far from the threshold (fp32 error is about 1e-6)
    acc = [fo[k] / (fo[k - 1] * (1 + tol)) - 1.0 for k in range(1, len(fo))]
    assert max(acc) < -2e-4, acc
    for t, eta, f in rej:  # each rejected attempt against the accepted objective before it
        assert f / (fo[t] * (1 + tol)) - 1.0 > 5e-4
    assert len(rej) >= 3
    _say("guard", m, n, "tol", tol, "oracle eta", eta_o, "rejected", len(rej))
    ctx = _ctx(m, n, r, blk, row_ptr, col, val, nmd.FLAG_GUARD, eta=1.0, mom=0.9, tol=tol,
               eta_min=1e-3)
    W, H = dev(W0), dev(H0)
    ctx.sweep(W, H, sweeps)
    eta_g, nrej = ctx.step_size()
    f = ctx.sweep_objectives()
    print(f"eta {eta_g} (oracle {eta_o}), rejected {nrej} (oracle {len(rej)})")
    print("f gpu   ", np.round(f, 6))
    print("f oracle", np.round(fo, 6))
    assert eta_g == eta_o and nrej == len(rej)
    assert ctx.sweep_count == sweeps
    assert np.max(np.abs(f - fo) / np.asarray(fo)) <= TOL
    ew, eh = rel(W.cpu().numpy(), st.W), rel(H.cpu().numpy(), st.H)
    print(f"rel err W {ew:.2e} H {eh:.2e}")
    assert ew <= TOL and eh <= TOL
    # the accepted objectives never rise by more than the tolerance
    assert all(f[k] <= f[k - 1] * (1 + tol) for k in range(1, len(f)))


def test_guard_floor_returns_estep_with_factors_before_the_sweep():
    """A step-size floor above the first halving's result: the first sweep is rejected at
    eta = 1 (eta -> 0.5), then again at 0.5; halving to 0.25 would cross eta_min = 0.3, so the
    call fails with NMD_ESTEP and W, H come back exactly as given (no sweep was accepted), the
    sweep counter stays at 0 and eta stays at 0.5."""
    m, n, r, blk = 240, 200, 8, 20
    row_ptr, col, val, W0, H0 = _problem(m, n, r, 0.1, 6)
    _say("guard floor")
    ctx = _ctx(m, n, r, blk, row_ptr, col, val, nmd.FLAG_GUARD, eta=1.0, mom=0.9, eta_min=0.3)
    W, H = dev(W0), dev(H0)
    with pytest.raises(nmd.NmdError) as e:
        ctx.sweep(W, H, 4)
    assert e.value.code == nmd.ESTEP
    assert np.array_equal(W.cpu().numpy(), W0) and np.array_equal(H.cpu().numpy(), H0)
    assert ctx.sweep_count == 0
    assert ctx.step_size() == (0.5, 2)
    ctx.reset()
    assert ctx.step_size() == (1.0, 0)


def test_guard_without_rises_is_the_plain_trajectory():
    """With a step size that never raises the objective, the safeguard changes nothing: the
    factors are bit-identical to the unguarded run."""
    m, n, r, blk = 300, 260, 8, 64
    row_ptr, col, val, W0, H0 = _problem(m, n, r, 0.08, 2)
    _say("guard, no rise")
    a = _ctx(m, n, r, blk, row_ptr, col, val, nmd.FLAG_GUARD, eta=0.5, tol=0.05)
    b = _ctx(m, n, r, blk, row_ptr, col, val, 0, eta=0.5)
    Wa, Ha, Wb, Hb = dev(W0), dev(H0), dev(W0), dev(H0)
    a.sweep(Wa, Ha, 3)
    b.sweep(Wb, Hb, 3)
    assert a.step_size() == (0.5, 0)
    assert np.array_equal(Wa.cpu().numpy(), Wb.cpu().numpy())
    assert np.array_equal(Ha.cpu().numpy(), Hb.cpu().numpy())


def test_sweep_counter_counts_completed_sweeps_after_a_rejected_step():
    """A singular Gram matrix in the first step of the second sweep: the call fails with
    NMD_ENOTPD after one completed sweep, so the counter reads 1, and the next call starts with
    the block order of sweep 1."""
    p = gen.config(1)
    p.mode = "stochastic"
    _say("counter after rejection")
    ctx = nmd.Context(p.m, p.n, p.r, p.block_m, p.block_n, seed=p.seed, mode="stochastic")
    ctx.set_sparse_csr(p.row_ptr, p.col, p.val)
    W, H = dev(p.W0), dev(p.H0)
    ctx.sweep(W, H, 1)
    code = ctx.schedule(1)[0]
    Hz = H.clone()
    if code > 0:  # zero the panel of sweep 1's first step: its Gram matrix is singular
        b = ctx.block_bounds(0)
        Hz[:, b[code - 1]:b[code]] = 0.0
    else:
        b = ctx.block_bounds(1)
        W[b[-code - 1]:b[-code], :] = 0.0
    with pytest.raises(nmd.NmdError) as e:
        ctx.sweep(W, Hz, 3)
    assert e.value.code == nmd.ENOTPD and "sweep 1, step 0" in e.value.message
    assert ctx.sweep_count == 1


def test_deterministic_rejection_keeps_factors_and_counter():
    """Deterministic mode (the exact half-steps): after one sweep, a zero H makes the next W
    half-step's Gram matrix singular.  The call fails with NMD_ENOTPD at sweep 1, step 0; W and H
    come back as they were passed, and the counter reads 1."""
    p = gen.config(1)  # deterministic
    _say("deterministic rejection")
    ctx = nmd.Context(p.m, p.n, p.r, p.block_m, p.block_n, seed=p.seed, mode="deterministic")
    ctx.set_sparse_csr(p.row_ptr, p.col, p.val)
    W, H = dev(p.W0), dev(p.H0)
    ctx.sweep(W, H, 1)
    W1 = W.clone()
    H.zero_()
    with pytest.raises(nmd.NmdError) as e:
        ctx.sweep(W, H, 2)
    assert e.value.code == nmd.ENOTPD and "sweep 1, step 0" in e.value.message
    assert ctx.sweep_count == 1
    assert torch.equal(W, W1) and not torch.any(H != 0).item()


def test_guard_in_deterministic_mode():
    """The safeguard with the deterministic half-steps (eqs. spLsqA, spLsqB) at an over-long step
    (eta = 1.7, momentum 0.9): sweeps 1 and 5 raise the objective in the oracle and are undone;
    the GPU makes the same decisions (a sweep is the two half-steps here, so the step ids of a
    sweep differ from the stochastic ones)."""
    m, n, r, blk, sweeps = 300, 260, 12, 64, 6
    row_ptr, col, val, W0, H0 = _problem(m, n, r, 0.1, 7)
    S = salsa.csr_matrix(m, n, row_ptr, col, val)
    st = salsa.State(W0, H0)
    eta_o, fo, rej = salsa.guarded_sweeps(S, S.T.tocsr(), st, blk, blk, 3, sweeps,
                                          "deterministic", 1.7, 0.9, eta_min=1e-3)
    assert [t for t, _, _ in rej] == [1, 5]
    assert min(f / fo[t] - 1.0 for t, _, f in rej) > 2e-3
    assert max(fo[k] / fo[k - 1] - 1.0 for k in range(1, len(fo))) < -1e-2
    _say("guard, deterministic mode")
    ctx = _ctx(m, n, r, blk, row_ptr, col, val, nmd.FLAG_GUARD, eta=1.7, mom=0.9, eta_min=1e-3,
               mode="deterministic")
    W, H = dev(W0), dev(H0)
    ctx.sweep(W, H, sweeps)
    f = ctx.sweep_objectives()
    print("f gpu   ", np.round(f, 6))
    print("f oracle", np.round(fo, 6))
    assert ctx.step_size() == (np.float32(eta_o), len(rej))
    assert np.max(np.abs(f - fo) / np.asarray(fo)) <= TOL
    assert rel(W.cpu().numpy(), st.W) <= TOL and rel(H.cpu().numpy(), st.H) <= TOL
