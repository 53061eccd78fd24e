"""Seeded synthetic inputs for subzero matrix completion, shared by the tests and the benchmark.

This module only draws inputs: sparse nonnegative matrices S in CSR form and initial factors
W (m x r), H (r x n).  It holds none of the method's arithmetic (no Z-update, no least-squares
step, no objective); the fp64 oracle and the GPU library each implement those on their own.

Every generator is a pure function of its arguments and seed (numpy PCG64).
"""

from .gen import (  # noqa: F401
    Problem,
    planted,
    identity,
    identity_exact_factors,
    graph_powerlaw,
    cooccurrence_zipf,
    random_sparse,
    sign_constrained_init,
    gaussian_init,
    config,
    CONFIGS,
)
