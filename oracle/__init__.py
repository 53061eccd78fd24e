"""Plain fp64 CPU oracle for stochastic alternating least squares in subzero matrix completion.

TEST INFRASTRUCTURE ONLY.  The tests, the smoke check and the CPU-baseline leg of the
benchmark call it; the GPU library never imports, links or executes it, and it shares no code
with the GPU path (kernels, headers, tables or helpers).

Contents:
  partition  balanced row/column block partition (a reading: the paper leaves it open)
  schedule   seeded per-sweep block order: SplitMix64, Lemire's bounded integers,
             Fisher-Yates shuffles and a proportional W/H interleave
  salsa      the method: rectification (eq. rectify), Z-update (eq. updateZ), the difference
             matrix (eq. updateD), least-squares, blockwise and stochastic updates
             (eqs. lsqA/lsqB, spLsqA/spLsqB, lsqA_par, Shat_sto/Delta_sto/lsqA_sto) with a
             heavy-ball momentum term, the objective (eqs. auxCost and SLloss), RMSE and WJD
             (eqs. RMSE, WJD).

Every routine computes in float64 from the float32 inputs the GPU receives (exact upcasts).
Parity pins: every function here is pinned by a CPU test against closed forms, invariants,
textbook routines or brute force (tests/test_oracle_pins.py, tests/test_schedule.py); none is
"parity unpinned".
"""

from . import partition, schedule, salsa  # noqa: F401
