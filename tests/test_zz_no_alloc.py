"""GPU: the allocation-free split-bf16 contraction (workspace in a static device array) against
the entry point that takes a caller-owned workspace: bit-identical outputs on consecutive calls,
the second smaller than the first, then a call at the workspace's limit and one beyond it."""

import ctypes as C

import numpy as np
import pytest
import torch

import paper_2608_21607_amd as nmd

pytestmark = pytest.mark.gpu

LIMIT_FLOATS = 4 << 20  # the static workspace (16 MiB)


def _noalloc():
    fn = nmd.lib().nmd_rectified_contraction_bf16x3_noalloc
    fn.restype = C.c_int32
    fn.argtypes = [C.c_void_p, C.c_int64, C.c_void_p, C.c_int64, C.c_int32, C.c_void_p,
                   C.c_void_p]
    return fn


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _case(fn, rows, blk, r, seed):
    print(f"[case] no-alloc contraction rows {rows} blk {blk} r {r}", flush=True)
    g = torch.Generator(device="cuda").manual_seed(seed)
    A = torch.randn((rows, r), generator=g, device="cuda")
    B = torch.randn((blk, r), generator=g, device="cuda")
    Y_ref = torch.full((rows, r), float("nan"), device="cuda")
    work = torch.empty((nmd.bf16x3_workspace_floats(blk, r),), device="cuda")
    nmd.rectified_contraction_bf16x3(A, B, Y_ref, work=work)
    Y = torch.full((rows, r), float("nan"), device="cuda")
    rc = fn(A.data_ptr(), rows, B.data_ptr(), blk, r, Y.data_ptr(), _stream())
    assert rc == 0, nmd.lib().nmd_last_error(None)
    torch.cuda.synchronize()
    assert torch.isfinite(Y).all()
    assert torch.equal(Y, Y_ref)
    # and the product itself, on sampled rows in fp64
    idx = torch.arange(0, rows, max(1, rows // 16), device="cuda")
    A64, B64 = A[idx].double(), B.double()
    want = torch.clamp(A64 @ B64.T, min=0.0) @ B64
    err = float(torch.linalg.norm(Y[idx].double() - want) / torch.linalg.norm(want))
    print(f"  bit-identical to the workspace form; sampled rel err vs fp64 {err:.2e}")
    assert err < 1e-4


def test_no_alloc_matches_workspace_form_on_consecutive_calls():
    fn = _noalloc()
    _case(fn, 1000, 4096, 256, 1)    # 1M floats of workspace
    _case(fn, 300, 700, 128, 2)      # smaller, after the larger one left its contents
    _case(fn, 257, 8192, 512, 3)     # exactly the static workspace's size at r = 512
    assert nmd.bf16x3_workspace_floats(8192, 512) == LIMIT_FLOATS


def test_no_alloc_rejects_a_panel_beyond_the_workspace():
    fn = _noalloc()
    print("[case] no-alloc contraction beyond the static workspace", flush=True)
    A = torch.zeros((16, 512), device="cuda")
    B = torch.zeros((8193, 512), device="cuda")
    Y = torch.zeros((16, 512), device="cuda")
    rc = fn(A.data_ptr(), 16, B.data_ptr(), 8193, 512, Y.data_ptr(), _stream())
    assert rc == nmd.EINVAL
    assert b"static workspace" in nmd.lib().nmd_last_error(None)
    rc = fn(A.data_ptr(), 16, B.data_ptr(), 10, 48, Y.data_ptr(), _stream())
    assert rc == nmd.EINVAL
