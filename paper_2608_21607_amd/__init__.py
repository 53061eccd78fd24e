"""MI355X (gfx950) stochastic alternating least squares for subzero matrix completion.

The method lives in libnmd.so (HIP kernels behind the C ABI of include/nmd.h); `nmd` is its
ctypes binding and `build` compiles it in-tree.
"""

from .nmd import (  # noqa: F401
    Context, NmdError, rectified_contraction, rectified_contraction_bf16x3,
    bf16x3_workspace_floats, lib,
    header_functions, DETERMINISTIC, STOCHASTIC, FLAG_ASYNC, FLAG_TIMING, FLAG_SPLIT_BF16,
    FLAG_SWEEP_OBJECTIVE, FLAG_GUARD, KERNEL_DENSE, KERNEL_SPARSE, KERNEL_FACTOR, KERNEL_APPLY,
    OK, EINVAL, ENOMEM, EDEVICE, ENOTPD, ESTATE, ENONFINITE, ESTEP,
)
