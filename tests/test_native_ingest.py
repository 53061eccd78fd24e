"""The library's host-only ingest code (schedule, partition, CSR validation, per-block arrays;
paper_2608_21607_amd/csrc/ingest.cpp) built with g++ under the address and undefined-behaviour
sanitizers and run on the CPU: structural invariants checked inside the driver
(tests/native/ingest_check.cpp), per-block entry counts against numpy, the block order against
the oracle's schedule, and the rejection of malformed matrices."""

import json
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import partition, schedule
from workloads import gen

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = [os.path.join(HERE, "native", "ingest_check.cpp"),
       os.path.join(ROOT, "paper_2608_21607_amd", "csrc", "ingest.cpp")]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("native") / "ingest_check")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-Wall", "-Werror",
           *SRC, "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return exe


def _run(exe, *args):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    res = subprocess.run([exe, *args], capture_output=True, text=True, env=env, timeout=600)
    assert res.returncode == 0, res.stdout[-2000:] + res.stderr[-4000:]
    assert "runtime error" not in res.stderr, res.stderr[-4000:]
    return json.loads(res.stdout)


def _ingest(exe, tmp_path, m, n, row_ptr, col, val, bm, bn):
    f = tmp_path / "in.bin"
    with open(f, "wb") as fh:
        np.array([m, n, len(col), bm, bn], dtype=np.int64).tofile(fh)
        np.asarray(row_ptr, dtype=np.int64).tofile(fh)
        np.asarray(col, dtype=np.int32).tofile(fh)
        np.asarray(val, dtype=np.float32).tofile(fh)
    return _run(exe, str(f))


def _expected_counts(m, n, row_ptr, col, val, bm, bn):
    rows = np.repeat(np.arange(m), np.diff(row_ptr))
    pos = np.asarray(val) > 0
    cb = np.array(partition.bounds(n, bn))
    rb = np.array(partition.bounds(m, bm))
    w = np.bincount(np.searchsorted(cb, np.asarray(col)[pos], "right") - 1, minlength=len(cb) - 1)
    h = np.bincount(np.searchsorted(rb, rows[pos], "right") - 1, minlength=len(rb) - 1)
    return w.tolist(), h.tolist()


def _case(exe, tmp_path, m, n, row_ptr, col, val, bm, bn):
    out = _ingest(exe, tmp_path, m, n, row_ptr, col, val, bm, bn)
    assert "error" not in out, out
    w, h = _expected_counts(m, n, row_ptr, col, val, bm, bn)
    assert out["w"]["nnz"] == w and out["h"]["nnz"] == h
    v = np.asarray(val, dtype=np.float32).astype(np.float64)  # what the driver receives
    assert abs(out["s2"] - float(np.sum(v[v > 0] ** 2))) <= 1e-9 * out["s2"]
    return out


def test_random_matrices_with_empty_rows_and_explicit_zeros(driver, tmp_path):
    for seed, (m, n, d, bm, bn) in enumerate([(1, 1, 1.0, 1, 1), (37, 53, 0.2, 7, 11),
                                               (300, 40, 0.05, 64, 16), (64, 900, 0.3, 64, 100)]):
        row_ptr, col, val = gen.random_sparse(m, n, d, seed)
        val = val.copy()
        val[::7] = 0.0  # explicit zeros are dropped
        if val.max() <= 0:
            continue
        _case(driver, tmp_path, m, n, row_ptr, col, val, bm, bn)


def test_heavy_row_is_split_into_items(driver, tmp_path):
    """One row holding half of the entries (far more than one item's worth per block)."""
    m, n = 50, 4000
    rng = np.random.default_rng(3)
    cols = [np.arange(0, n, 2)] + [np.sort(rng.choice(n, 20, replace=False)) for _ in range(m - 1)]
    row_ptr = np.concatenate([[0], np.cumsum([len(c) for c in cols])])
    col = np.concatenate(cols)
    val = rng.uniform(0.5, 2.0, col.size)
    out = _case(driver, tmp_path, m, n, row_ptr, col, val, 16, 1000)
    assert out["w"]["splits"] == 4 and out["w"]["max_slots"] == 4  # 500 entries per block


@pytest.mark.parametrize("k,scale", [(4, 0.1), (5, 0.01)])
def test_workload_generators(driver, tmp_path, k, scale):
    """The graph workload (power-law rows) and the co-occurrence workload (Zipf rows, the
    heaviest fully dense) at reduced size, with their block sizes."""
    p = gen.config(k, scale)
    out = _case(driver, tmp_path, p.m, p.n, p.row_ptr, p.col, p.val, p.block_m, p.block_n)
    assert out["w"]["items"] >= len(out["w"]["nnz"])


def test_schedule_matches_oracle(driver):
    for seed, t, R, C in [(4, 0, 17, 17), (5, 3, 31, 7), (2**63 + 5, 11, 1, 9), (1, 0, 1, 1)]:
        out = _run(driver, "--schedule", str(seed), str(t), str(R), str(C))
        assert out["schedule"] == schedule.sweep_schedule(seed, t, R, C, True)


@pytest.mark.parametrize("bad,msg", [
    ("unsorted", "not strictly increasing"), ("duplicate", "not strictly increasing"),
    ("negative", "negative or not finite"), ("nan", "negative or not finite"),
    ("range", "out of range"), ("ptr0", "row_ptr[0]"), ("ptrdec", "decreases"),
    ("ptrend", "differs from nnz"), ("zeros", "no positive entry")])
def test_malformed_matrices_are_rejected(driver, tmp_path, bad, msg):
    m, n = 6, 8
    row_ptr = np.array([0, 2, 3, 3, 5, 6, 7])
    col = np.array([1, 4, 0, 2, 7, 5, 6])
    val = np.ones(7)
    if bad == "unsorted":
        col[[0, 1]] = [4, 1]
    elif bad == "duplicate":
        col[1] = 1
    elif bad == "negative":
        val[3] = -1.0
    elif bad == "nan":
        val[5] = np.nan
    elif bad == "range":
        col[6] = 8
    elif bad == "ptr0":
        row_ptr = row_ptr + 1
    elif bad == "ptrdec":
        row_ptr[2] = 1
    elif bad == "ptrend":
        row_ptr[-1] = 6
    elif bad == "zeros":
        val[:] = 0.0
    out = _ingest(driver, tmp_path, m, n, row_ptr, col, val, 3, 3)
    assert msg in out.get("error", ""), out
