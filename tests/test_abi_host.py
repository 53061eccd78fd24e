"""The C ABI without a GPU: exported symbols, argument validation, block partition, the block
schedule (bit-exact against the oracle) and the per-block nonzero counts.  No call here reaches
the device."""

import ctypes as C
import json
import os

import numpy as np
import pytest

from oracle import partition, schedule
from workloads import gen

nmd = pytest.importorskip("paper_2608_21607_amd.nmd")

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(nmd.LIB_PATH):
        pytest.skip("libnmd.so not built")
    return nmd.lib()


def test_every_declared_symbol_is_exported(L):
    names = nmd.header_functions()
    assert len(names) >= 14
    for name in names:
        assert hasattr(L, name), name
    for core in ("nmd_create", "nmd_set_sparse_csr", "nmd_als_block_sweep", "nmd_objective",
                 "nmd_destroy"):
        assert core in names


def _create(m, n, r, bm, bn, seed=1, mode=nmd.STOCHASTIC, eta=1.0, mom=0.0, size=None, flags=0,
            guard_tol=0.0, eta_min=0.0):
    opts = nmd.Options(C.sizeof(nmd.Options) if size is None else size, mode, eta, mom, flags,
                       guard_tol, eta_min)
    p = C.c_void_p()
    rc = nmd.lib().nmd_create(C.byref(p), m, n, r, bm, bn, seed, C.byref(opts))
    return rc, p


@pytest.mark.parametrize("args", [
    (0, 10, 1, 4, 4), (10, 0, 1, 4, 4), (10, 10, 0, 4, 4), (10, 10, 11, 4, 4),
    (1000, 1000, 513, 999, 999), (10, 10, 2, 0, 4), (10, 10, 2, 4, 0),
    (100, 100, 30, 25, 100),  # rank above the smallest row block in stochastic mode
])
def test_create_rejects_bad_sizes(L, args):
    rc, p = _create(*args)
    assert rc == nmd.EINVAL and not p.value
    assert L.nmd_last_error(None)


def test_create_rejects_bad_options(L):
    assert _create(10, 10, 2, 5, 5, mode=7)[0] == nmd.EINVAL
    assert _create(10, 10, 2, 5, 5, eta=float("nan"))[0] == nmd.EINVAL
    assert _create(10, 10, 2, 5, 5, mom=1.0)[0] == nmd.EINVAL
    assert _create(10, 10, 2, 5, 5, size=4)[0] == nmd.EINVAL
    assert _create(10, 10, 2, 5, 5, flags=32)[0] == nmd.EINVAL  # unknown option flag
    assert _create(10, 10, 2, 5, 5, guard_tol=-0.1)[0] == nmd.EINVAL
    assert _create(10, 10, 2, 5, 5, eta_min=float("inf"))[0] == nmd.EINVAL
    assert _create(10, 10, 2, 5, 5, size=16)[0] == nmd.EINVAL  # shorter than five fields
    for f in (nmd.FLAG_ASYNC, nmd.FLAG_TIMING, nmd.FLAG_SPLIT_BF16, nmd.FLAG_SWEEP_OBJECTIVE,
              nmd.FLAG_GUARD):
        rc, p = _create(10, 10, 2, 5, 5, flags=f)
        assert rc == 0
        L.nmd_destroy(p)
    # a caller of the five-field options struct (size 20) is accepted, later fields default
    rc, p = _create(10, 10, 2, 5, 5, size=20, eta=0.5)
    assert rc == 0
    eta = C.c_float()
    rej = C.c_int64(7)
    assert L.nmd_get_step_size(p, C.byref(eta), C.byref(rej)) == 0
    assert eta.value == 0.5 and rej.value == 0
    L.nmd_destroy(p)
    # deterministic mode accepts r above the block size
    rc, p = _create(100, 100, 30, 25, 25, mode=nmd.DETERMINISTIC)
    assert rc == 0
    L.nmd_destroy(p)
    L.nmd_destroy(None)


def _csr_case():
    row_ptr = np.array([0, 2, 2, 5], dtype=np.int64)
    col = np.array([1, 3, 0, 2, 3], dtype=np.int32)
    val = np.array([1.0, 2.0, 0.5, 0.0, 3.0], dtype=np.float32)
    return row_ptr, col, val


@pytest.mark.parametrize("mutate,msg", [
    (lambda rp, c, v: rp.__setitem__(0, 1), "row_ptr[0]"),
    (lambda rp, c, v: rp.__setitem__(2, 6), "decreases"),
    (lambda rp, c, v: rp.__setitem__(3, 4), "row_ptr[m]"),
    (lambda rp, c, v: c.__setitem__(1, 1), "strictly increasing"),
    (lambda rp, c, v: c.__setitem__(4, 2), "strictly increasing"),
    (lambda rp, c, v: c.__setitem__(0, 4), "out of range"),
    (lambda rp, c, v: c.__setitem__(0, -1), "out of range"),
    (lambda rp, c, v: v.__setitem__(0, -1.0), "negative"),
    (lambda rp, c, v: v.__setitem__(0, np.nan), "not finite"),
    (lambda rp, c, v: v.__setitem__(0, np.inf), "not finite"),
])
def test_csr_validation(L, mutate, msg):
    ctx = nmd.Context(3, 4, 1, 2, 2, mode="stochastic")
    rp, c, v = _csr_case()
    ctx.set_sparse_csr(rp, c, v)  # valid
    mutate(rp, c, v)
    with pytest.raises(nmd.NmdError) as e:
        ctx.set_sparse_csr(rp, c, v)
    assert e.value.code == nmd.EINVAL and msg in e.value.message
    ctx.close()


def test_no_positive_entry_and_state_errors(L):
    ctx = nmd.Context(3, 4, 1, 2, 2)
    with pytest.raises(nmd.NmdError) as e:
        ctx.set_sparse_csr(np.zeros(4, np.int64), np.zeros(0, np.int32), np.zeros(0, np.float32))
    assert e.value.code == nmd.EINVAL
    with pytest.raises(nmd.NmdError) as e:
        ctx.set_sparse_csr([0, 1, 1, 1], [2], [0.0])
    assert e.value.code == nmd.EINVAL
    fake = C.c_void_p(0x1000)
    assert L.nmd_als_block_sweep(ctx._p, fake, fake, 1, None) == nmd.ESTATE
    assert L.nmd_als_block_sweep(ctx._p, None, fake, 1, None) == nmd.EINVAL
    out = C.c_double()
    assert L.nmd_objective(ctx._p, fake, fake, C.byref(out), None) == nmd.ESTATE
    out3 = (C.c_double * 3)()
    assert L.nmd_metrics(ctx._p, fake, fake, out3, None) == nmd.ESTATE
    assert L.nmd_metrics(None, fake, fake, out3, None) == nmd.EINVAL
    ctx.set_sparse_csr(*_csr_case())
    assert L.nmd_metrics(ctx._p, fake, fake, None, None) == nmd.EINVAL
    assert L.nmd_metrics(ctx._p, None, fake, out3, None) == nmd.EINVAL
    assert L.nmd_als_block_sweep(ctx._p, fake, fake, 0, None) == nmd.EINVAL
    # a call enqueues at most 2^27 steps (the device status word holds step id * 8 + flag);
    # 2 x 2 blocks make 4 steps per sweep.  Rejected before the device or the list is touched.
    assert L.nmd_als_block_sweep(ctx._p, fake, fake, (1 << 25) + 1, None) == nmd.EINVAL
    assert "split the call" in nmd.lib().nmd_last_error(ctx._p).decode()
    one = (C.c_int32 * 1)(1)
    assert L.nmd_run_steps(ctx._p, fake, fake, one, (1 << 27) + 1, None) == nmd.EINVAL
    steps = (C.c_int32 * 1)(3)
    assert L.nmd_run_steps(ctx._p, fake, fake, steps, 1, None) == nmd.EINVAL
    steps = (C.c_int32 * 1)(0)
    assert L.nmd_run_steps(ctx._p, fake, fake, steps, 1, None) == nmd.EINVAL
    assert L.nmd_objective(ctx._p, fake, fake, None, None) == nmd.EINVAL
    ctx.close()


def test_rectified_contraction_argument_checks(L):
    fake = C.c_void_p(0x1000)
    for r in (8, 17, 80, 96, 576):
        assert L.nmd_rectified_contraction(fake, 10, fake, 10, r, fake, None) == nmd.EINVAL
    assert L.nmd_rectified_contraction(fake, 0, fake, 10, 16, fake, None) == nmd.EINVAL
    assert L.nmd_rectified_contraction(fake, 10, fake, 0, 16, fake, None) == nmd.EINVAL
    assert L.nmd_rectified_contraction(None, 10, fake, 10, 16, fake, None) == nmd.EINVAL
    bx = L.nmd_rectified_contraction_bf16x3
    for r in (8, 48, 96, 192, 384, 1024):  # both-products bf16: r in 16, 32, 64, 128, 256, 512
        assert bx(fake, 10, fake, 10, r, fake, fake, None) == nmd.EINVAL
    assert bx(fake, 10, fake, 10, 64, None, fake, None) == nmd.EINVAL
    assert bx(fake, 10, fake, 0, 64, fake, fake, None) == nmd.EINVAL


def test_bf16x3_workspace_size(L):
    """blk r + 32 ceil(blk / 32) max(r, 32) floats at r <= 128: the row-major copy and the
    pair-padded, at least 32-column transposed copy; blk r at r = 256 and 512 (row-major only)."""
    for blk, r in ((1, 16), (40, 16), (1, 32), (31, 64), (32, 64), (33, 128), (2500, 128)):
        assert nmd.bf16x3_workspace_floats(blk, r) == blk * r + 32 * ((blk + 31) // 32) * max(r, 32)
    for blk, r in ((1, 256), (8192, 256), (33, 512), (50000, 512)):
        assert nmd.bf16x3_workspace_floats(blk, r) == blk * r
    assert nmd.bf16x3_workspace_floats(0, 64) == -1
    assert nmd.bf16x3_workspace_floats(10, 8) == -1
    assert nmd.bf16x3_workspace_floats(10, 384) == -1


def test_dense_blocks_before_device_use(L):
    """The skip counters of a context that has not touched the GPU read zero."""
    ctx = nmd.Context(40, 30, 4, 16, 16)
    assert ctx.dense_blocks() == (0, 0, 0)
    assert L.nmd_get_dense_blocks(None, None, None, None, 0) == nmd.EINVAL
    ctx.close()


def test_kernel_timing_classes_before_device_use(L):
    """Five timing classes (dense, sparse, Gram and inverse, update, wait for the side stream)
    read zero before any work; a sixth is rejected."""
    ctx = nmd.Context(40, 30, 4, 16, 16)
    for k in range(5):
        assert ctx.kernel_timing(k) == {"ms": 0.0, "launches": 0, "flops": 0.0, "bytes": 0.0}
    ms = C.c_double()
    assert L.nmd_get_kernel_timing(ctx._p, 5, C.byref(ms), None, None, None, 0) == nmd.EINVAL
    assert L.nmd_get_kernel_timing(ctx._p, -1, C.byref(ms), None, None, None, 0) == nmd.EINVAL
    ctx.close()


def test_schedule_matches_golden_and_oracle(L):
    with open(os.path.join(HERE, "golden", "schedules.json")) as f:
        cases = json.load(f)
    for case in cases:
        ctx = nmd.Context(case["m"], case["n"], 1, case["block_m"], case["block_n"],
                          seed=int(case["seed"]), mode="stochastic")
        assert ctx.block_bounds(1).tolist() == case["row_bounds"]
        assert ctx.block_bounds(0).tolist() == case["col_bounds"]
        assert ctx.schedule(case["sweep"]) == case["steps"]
        ctx.close()
    rng = np.random.default_rng(0)
    for _ in range(40):
        m, n = (int(x) for x in rng.integers(1, 3000, 2))
        bm, bn = (int(x) for x in rng.integers(1, 400, 2))
        seed = int(rng.integers(0, 2**63)) * 2 + 1
        t = int(rng.integers(0, 1000))
        ctx = nmd.Context(m, n, 1, bm, bn, seed=seed, mode="stochastic")
        R, Cn = partition.num_blocks(m, bm), partition.num_blocks(n, bn)
        assert ctx.schedule(t) == schedule.sweep_schedule(seed, t, R, Cn, True)
        assert ctx.block_bounds(1).tolist() == partition.bounds(m, bm)
        ctx.close()
    ctx = nmd.Context(50, 40, 2, 7, 9, seed=5, mode="deterministic")
    assert ctx.schedule(3) == schedule.sweep_schedule(5, 3, 8, 5, False)
    ctx.close()


def test_block_nnz_counts_match_numpy(L):
    p = gen.config(1)
    ctx = nmd.Context(p.m, p.n, p.r, p.block_m, p.block_n, mode="stochastic")
    val = p.val.copy()
    val[::7] = 0.0  # explicit zeros are dropped
    ctx.set_sparse_csr(p.row_ptr, p.col, val)
    rows, cols, _ = p.coo()
    keep = val > 0
    rb = np.array(partition.bounds(p.m, p.block_m))
    cb = np.array(partition.bounds(p.n, p.block_n))
    want_c = np.bincount(np.searchsorted(cb, cols[keep], side="right") - 1, minlength=len(cb) - 1)
    want_r = np.bincount(np.searchsorted(rb, rows[keep], side="right") - 1, minlength=len(rb) - 1)
    assert ctx.block_nnz(0).tolist() == want_c.tolist()
    assert ctx.block_nnz(1).tolist() == want_r.tolist()
    ctx.close()
