"""ctypes binding of libnmd (include/nmd.h): argument marshalling only.

Every step of the method runs in the HIP kernels of libnmd.so; this module converts numpy
arrays and torch tensors to pointers and sizes and turns status codes into exceptions.
PyTorch supplies device memory and streams.  If the library has not been built the calls fail
loudly; there is no fallback path.
"""

from __future__ import annotations

import ctypes as C
import os
import re

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libnmd.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "nmd.h")

OK, EINVAL, ENOMEM, EDEVICE, ENOTPD, ESTATE, ENONFINITE, ESTEP = 0, -1, -2, -3, -4, -5, -6, -7
CODE_NAMES = {0: "NMD_OK", -1: "NMD_EINVAL", -2: "NMD_ENOMEM", -3: "NMD_EDEVICE",
              -4: "NMD_ENOTPD", -5: "NMD_ESTATE", -6: "NMD_ENONFINITE", -7: "NMD_ESTEP"}
DETERMINISTIC, STOCHASTIC = 0, 1
FLAG_ASYNC, FLAG_TIMING, FLAG_SPLIT_BF16, FLAG_SWEEP_OBJECTIVE, FLAG_GUARD = 1, 2, 4, 8, 16
KERNEL_DENSE, KERNEL_SPARSE, KERNEL_FACTOR, KERNEL_APPLY = 0, 1, 2, 3


class NmdError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{CODE_NAMES.get(code, code)}: {message}")
        self.code = code
        self.message = message


class Options(C.Structure):
    _fields_ = [("size", C.c_uint32), ("mode", C.c_int32), ("eta", C.c_float),
                ("momentum", C.c_float), ("flags", C.c_uint32), ("guard_tol", C.c_float),
                ("eta_min", C.c_float)]


_lib = None


def lib() -> C.CDLL:
    """The loaded libnmd.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2608_21607_amd.build` (no CPU fallback exists)")
    L = C.CDLL(LIB_PATH)
    P, I32, I64, U64, F = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_float
    sig = {
        "nmd_create": (I32, [C.POINTER(P), I64, I64, I32, I32, I32, U64, C.POINTER(Options)]),
        "nmd_set_sparse_csr": (I32, [P, I64, P, P, P]),
        "nmd_als_block_sweep": (I32, [P, P, P, I32, P]),
        "nmd_objective": (I32, [P, P, P, C.POINTER(C.c_double), P]),
        "nmd_metrics": (I32, [P, P, P, P, P]),
        "nmd_destroy": (None, [P]),
        "nmd_last_error": (C.c_char_p, [P]),
        "nmd_get_schedule": (I32, [P, I64, P, I64]),
        "nmd_get_block_nnz": (I32, [P, I32, P, I64]),
        "nmd_get_block_bounds": (I32, [P, I32, P, I64]),
        "nmd_reset": (I32, [P]),
        "nmd_get_sweep_count": (I32, [P, C.POINTER(I64)]),
        "nmd_get_sweep_objectives": (I32, [P, P, I64]),
        "nmd_get_step_size": (I32, [P, C.POINTER(F), C.POINTER(I64)]),
        "nmd_run_steps": (I32, [P, P, P, P, I32, P]),
        "nmd_rectified_contraction": (I32, [P, I64, P, I64, I32, P, P]),
        "nmd_rectified_contraction_bf16x3": (I32, [P, I64, P, I64, I32, P, P, P]),
        "nmd_bf16x3_workspace_floats": (I64, [I64, I32]),
        "nmd_get_dense_blocks": (I32, [P, P, P, P, I32]),
        "nmd_get_kernel_timing": (I32, [P, I32, C.POINTER(C.c_double), C.POINTER(I64),
                                        C.POINTER(C.c_double), C.POINTER(C.c_double), I32]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def header_functions(path: str = HEADER):
    """Names of the functions include/nmd.h declares."""
    with open(path) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(nmd_\w+)\s*\(", text)))


def _check(code: int, ctx_ptr=None):
    if code >= 0:
        return code
    msg = lib().nmd_last_error(ctx_ptr)
    raise NmdError(code, msg.decode() if msg else "")


def _stream_handle(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _dev_ptr(t, shape, name):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) torch tensor")
    if t.dtype != torch.float32 or not t.is_contiguous() or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must be a contiguous float32 tensor of shape {tuple(shape)}, "
                         f"got {t.dtype} {tuple(t.shape)} contiguous={t.is_contiguous()}")
    return C.c_void_p(t.data_ptr())


class Context:
    """An nmd_ctx: the problem sizes, S, the block partition and the optimiser state."""

    def __init__(self, m, n, r, block_m, block_n, seed=1, mode="deterministic", eta=1.0,
                 momentum=0.0, flags=0, guard_tol=0.0, eta_min=0.0):
        self._p = None
        md = {"deterministic": DETERMINISTIC, "stochastic": STOCHASTIC}.get(mode, mode)
        opts = Options(C.sizeof(Options), int(md), float(eta), float(momentum), int(flags),
                       float(guard_tol), float(eta_min))
        p = C.c_void_p()
        _check(lib().nmd_create(C.byref(p), int(m), int(n), int(r), int(block_m), int(block_n),
                                int(seed) & (2**64 - 1), C.byref(opts)), None)
        self._p = p
        self.m, self.n, self.r = int(m), int(n), int(r)

    def close(self):
        if self._p is not None and self._p.value:
            lib().nmd_destroy(self._p)
        self._p = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def set_sparse_csr(self, row_ptr, col, val):
        rp = np.ascontiguousarray(row_ptr, dtype=np.int64)
        ci = np.ascontiguousarray(col, dtype=np.int32)
        vv = np.ascontiguousarray(val, dtype=np.float32)
        nnz = int(ci.size)
        _check(lib().nmd_set_sparse_csr(self._p, nnz, rp.ctypes.data_as(C.c_void_p),
                                        ci.ctypes.data_as(C.c_void_p) if nnz else None,
                                        vv.ctypes.data_as(C.c_void_p) if nnz else None), self._p)

    def sweep(self, W, H, n_sweeps=1, stream=None):
        _check(lib().nmd_als_block_sweep(self._p, _dev_ptr(W, (self.m, self.r), "W"),
                                         _dev_ptr(H, (self.r, self.n), "H"), int(n_sweeps),
                                         _stream_handle(stream)), self._p)

    def sweep_objectives(self):
        """Objectives before and after each sweep of the last sweep call (NMD_FLAG_GUARD or
        NMD_FLAG_SWEEP_OBJECTIVE)."""
        cap = 1 << 16
        out = np.zeros(cap, dtype=np.float64)
        k = _check(lib().nmd_get_sweep_objectives(self._p, out.ctypes.data_as(C.c_void_p), cap),
                   self._p)
        return out[:k].copy()

    def step_size(self):
        """(eta now in force, number of sweeps the safeguard has undone)."""
        eta = C.c_float()
        rej = C.c_int64()
        _check(lib().nmd_get_step_size(self._p, C.byref(eta), C.byref(rej)), self._p)
        return float(eta.value), int(rej.value)

    def run_steps(self, W, H, steps, stream=None):
        s = np.ascontiguousarray(steps, dtype=np.int32)
        _check(lib().nmd_run_steps(self._p, _dev_ptr(W, (self.m, self.r), "W"),
                                   _dev_ptr(H, (self.r, self.n), "H"),
                                   s.ctypes.data_as(C.c_void_p), int(s.size),
                                   _stream_handle(stream)), self._p)

    def objective(self, W, H, stream=None) -> float:
        out = C.c_double()
        _check(lib().nmd_objective(self._p, _dev_ptr(W, (self.m, self.r), "W"),
                                   _dev_ptr(H, (self.r, self.n), "H"), C.byref(out),
                                   _stream_handle(stream)), self._p)
        return out.value

    def metrics(self, W, H, stream=None) -> dict:
        """Objective, RMSE and weighted Jaccard distance of S-hat = max(0, W H), one pass."""
        out = (C.c_double * 3)()
        _check(lib().nmd_metrics(self._p, _dev_ptr(W, (self.m, self.r), "W"),
                                 _dev_ptr(H, (self.r, self.n), "H"), out,
                                 _stream_handle(stream)), self._p)
        return {"objective": out[0], "rmse": out[1], "wjd": out[2]}

    def schedule(self, t):
        cap = 1 << 20
        buf = np.zeros(cap, dtype=np.int32)
        k = _check(lib().nmd_get_schedule(self._p, int(t), buf.ctypes.data_as(C.c_void_p), cap), self._p)
        return buf[:k].tolist()

    def block_nnz(self, side):
        buf = np.zeros(1 << 20, dtype=np.int64)
        k = _check(lib().nmd_get_block_nnz(self._p, int(side), buf.ctypes.data_as(C.c_void_p), buf.size), self._p)
        return buf[:k].copy()

    def block_bounds(self, side):
        buf = np.zeros(1 << 20, dtype=np.int64)
        k = _check(lib().nmd_get_block_bounds(self._p, int(side), buf.ctypes.data_as(C.c_void_p), buf.size), self._p)
        return buf[:k].copy()

    def reset(self):
        _check(lib().nmd_reset(self._p), self._p)

    @property
    def sweep_count(self) -> int:
        t = C.c_int64()
        _check(lib().nmd_get_sweep_count(self._p, C.byref(t)), self._p)
        return t.value

    def kernel_timing(self, kernel, reset=False):
        ms, n, fl, by = C.c_double(), C.c_int64(), C.c_double(), C.c_double()
        _check(lib().nmd_get_kernel_timing(self._p, int(kernel), C.byref(ms), C.byref(n),
                                           C.byref(fl), C.byref(by), int(bool(reset))), self._p)
        return {"ms": ms.value, "launches": n.value, "flops": fl.value, "bytes": by.value}

    def dense_blocks(self, reset=False):
        """(run, total, entries): slices (16 rows x 4 panel rows) of the dense contraction's
        second product that ran whole, slices examined, and positive entries taken through
        gathered slices, since creation or the last reset."""
        run, tot, ent = C.c_int64(), C.c_int64(), C.c_int64()
        _check(lib().nmd_get_dense_blocks(self._p, C.byref(run), C.byref(tot), C.byref(ent),
                                          int(bool(reset))), self._p)
        return run.value, tot.value, ent.value


def rectified_contraction(A, B, Y=None, stream=None):
    """Y = max(0, A B^T) B on the GPU (A: rows x r, B: blk x r, float32 CUDA tensors)."""
    import torch
    rows, r = A.shape
    blk = B.shape[0]
    if Y is None:
        Y = torch.empty((rows, r), dtype=torch.float32, device=A.device)
    _check(lib().nmd_rectified_contraction(_dev_ptr(A, (rows, r), "A"), int(rows),
                                           _dev_ptr(B, (blk, r), "B"), int(blk), int(r),
                                           _dev_ptr(Y, (rows, r), "Y"), _stream_handle(stream)),
           None)
    return Y


def bf16x3_workspace_floats(blk, r) -> int:
    """Floats of workspace rectified_contraction_bf16x3 needs (-1 for an unsupported r)."""
    return int(lib().nmd_bf16x3_workspace_floats(int(blk), int(r)))


def rectified_contraction_bf16x3(A, B, Y=None, work=None, stream=None):
    """Y = max(0, A B^T) B with both products on split bf16 MFMA (A: rows x r, B: blk x r,
    float32 CUDA tensors, r in {16, 32, 64, 128, 256, 512}; work: float32 workspace of at least
    bf16x3_workspace_floats(blk, r) elements)."""
    import torch
    rows, r = A.shape
    blk = B.shape[0]
    need = bf16x3_workspace_floats(blk, r)
    if need < 0:
        raise NmdError(EINVAL, f"the bf16x3 contraction needs r in (16, 32, 64, 128, 256, 512), got {r}")
    if Y is None:
        Y = torch.empty((rows, r), dtype=torch.float32, device=A.device)
    if work is None:
        work = torch.empty((need,), dtype=torch.float32, device=A.device)
    if not work.is_cuda or work.dtype != torch.float32 or not work.is_contiguous() or work.numel() < need:
        raise ValueError(f"work must be a contiguous float32 CUDA tensor of at least {need} elements")
    _check(lib().nmd_rectified_contraction_bf16x3(
        _dev_ptr(A, (rows, r), "A"), int(rows), _dev_ptr(B, (blk, r), "B"), int(blk), int(r),
        C.c_void_p(work.data_ptr()), _dev_ptr(Y, (rows, r), "Y"), _stream_handle(stream)), None)
    return Y
