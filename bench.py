"""Benchmark: stochastic ALS sweeps per second on one MI355X.

Default workload: the 139,255 x 139,255 graph-like count matrix with ~16.8M nonzeros
(power-law Chung-Lu sampler, 50 planted communities, lognormal counts), rank 256, blocks of
8192 x 8192, stochastic mode with step size 0.1 and momentum 0.9 (a synthetic stand-in for the
paper's connectome matrix).  A step of this benchmark is one full sweep: every column block
drives one W-step and every row block one H-step.  The objective after every sweep is recorded
from a second, untimed run of the same sweeps (the kernels are deterministic; its final factors
are checked to equal the timed run's), with the number of sweeps that raised it.

Prints one JSON line.  `value` is sweeps/s with every input resident in HBM.  `roofline`
reports the fused dense kernel (the dominant one) from HIP events recorded around each of its
launches on the stream it runs on.  `cpu_baseline` times the fp64 oracle on the host cores over
a bounded sample of the same workload (the first W-step and the first H-step of sweep 0 at full
size), scaled to sweeps/s.

    python bench.py [--steps K] [--warmup W] [--config 4] [--no-cpu-baseline]
    python bench.py --kernel-mb      (the fused kernel alone, shape of the paper's kernel table)
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP32_MFMA = 157.3   # TFLOP/s, MI355X dense fp32 matrix
PEAK_BF16_MFMA = 2500.0  # TFLOP/s, MI355X dense bf16 matrix
PEAK_HBM = 8.0e3         # GB/s, MI355X HBM3E

METRIC = "ALS sweeps/sec and dense-equiv TFLOP/s (4mnr/sweep), % of fp32 MFMA peak"

# HBM traffic of the fused dense kernel, from two rocprofv3 --pmc passes (FETCH_SIZE, then
# WRITE_SIZE) scaled by the same counters on a plain copy of known size; valid only for the
# kernel sources it was taken on.
_CSRC = os.path.join(ROOT, "paper_2608_21607_amd", "csrc")
_SPLIT_SOURCES = ("tile.h", "dense_kernel.h", "dense_bf16.h", "dense_bf16.hip", "dense_bf16_large.hip")
# (variant, workload) -> counter summary, and the sources of the dense kernel it measured
TRAFFIC_FILES = {
    ("fp32", 4): os.path.join(ROOT, "profiles", "dense_r256_graph139255_traffic.json"),
    ("split_bf16", 4): os.path.join(ROOT, "profiles", "bf16x3_r256_graph139255_traffic.json"),
    ("fp32", 5): os.path.join(ROOT, "profiles", "dense_r512_cooc500000x50000_traffic.json"),
    ("split_bf16", 5): os.path.join(ROOT, "profiles", "bf16x3_r512_cooc500000x50000_traffic.json"),
}
KERNEL_SOURCES = {
    ("fp32", 4): [os.path.join(_CSRC, f) for f in ("tile.h", "dense_kernel.h", "dense.hip")],
    ("split_bf16", 4): [os.path.join(_CSRC, f) for f in _SPLIT_SOURCES],
    ("fp32", 5): [os.path.join(_CSRC, f) for f in ("tile.h", "dense_kernel.h", "dense_large.hip")],
    ("split_bf16", 5): [os.path.join(_CSRC, f) for f in _SPLIT_SOURCES],
}


def kernel_source_hash(variant="fp32", config=4):
    """SHA-256 of the dense kernel's sources with // comments, trailing blanks and blank lines
    removed, so that it changes with the code and not with its comments."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[(variant, config)]:
        with open(f) as fh:
            for line in fh:
                code = re.sub(r"//.*", "", line).rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()


def measured_traffic(config, variant="fp32"):
    """Bytes per dense-kernel launch from the committed counter summary, or None when the
    summary is missing, was taken on another workload, or the kernel has changed since."""
    if (variant, config) not in TRAFFIC_FILES:
        return None
    try:
        with open(TRAFFIC_FILES[(variant, config)]) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if (t.get("kernel_source_sha256") != kernel_source_hash(variant, config)
            or t.get("config") != config):
        return None
    return t.get("traffic_bytes_per_launch")


# The paper's fused TF32 kernel at m = 250000 rows, a 2500-row panel (its kernel throughput
# table, Sec. 4.2): TFLOP/s on an H100 PCIe and on an RTX Pro 6000 Blackwell.  Context only:
# other hardware, and TF32 (gfx950 has no TF32 matrix instructions; the kernel here is fp32).
PAPER_FUSED_TF32 = {16: (215.30, 191.72), 32: (283.73, 203.06), 64: (285.10, 206.11),
                    128: (279.19, 189.80)}


def kernel_mb(steps, warmup):
    """The fused rectified contraction Y = max(0, A B^T) B alone at the shape of the paper's
    kernel table: A 250000 x r, B 2500 x r, N(0,1) entries.  About half of L is positive, so
    every slice of the second product runs and the work is 4 rows blk r flops.  Timed for the
    fp32 kernel and for the kernel with both products on split bf16 (bf16x3), at the paper's
    ranks 16 to 128 and at the workloads' ranks 256 and 512 (no paper figure there)."""
    import torch

    import paper_2608_21607_amd as nmd

    rows, blk = 250_000, 2500
    res = []
    for r in (16, 32, 64, 128, 256, 512):
        g = torch.Generator(device="cuda").manual_seed(r)
        A = torch.randn((rows, r), generator=g, device="cuda")
        B = torch.randn((blk, r), generator=g, device="cuda")
        Y = torch.empty((rows, r), device="cuda")
        runs = [("fp32", lambda: nmd.rectified_contraction(A, B, Y))]
        if nmd.bf16x3_workspace_floats(blk, r) > 0:
            work = torch.empty((nmd.bf16x3_workspace_floats(blk, r),), device="cuda")
            runs.append(("bf16x3", lambda: nmd.rectified_contraction_bf16x3(A, B, Y, work=work)))
        row = {"r": r}
        for tag, f in runs:
            for _ in range(warmup):
                f()
            start = torch.cuda.Event(enable_timing=True)
            stop = torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            start.record()
            for _ in range(steps):
                f()
            stop.record()
            torch.cuda.synchronize()
            ms = start.elapsed_time(stop) / steps
            tflops = 4.0 * rows * blk * r / (ms / 1e3) / 1e12
            if tag == "fp32":
                row.update({"ms_per_launch": ms, "tflops": tflops,
                            "frac_of_fp32_peak": tflops / PEAK_FP32_MFMA})
            else:
                row.update({"bf16x3_ms_per_launch": ms, "bf16x3_tflops": tflops,
                            "bf16x3_frac_of_peak": tflops / (PEAK_BF16_MFMA / 3.0)})
            log(f"r = {r} {tag}: {ms:.3f} ms per launch, {tflops:.1f} TFLOP/s")
        h100, rtx = PAPER_FUSED_TF32.get(r, (None, None))
        row.update({"paper_tf32_h100_pcie": h100, "paper_tf32_rtx_pro_6000": rtx})
        res.append(row)
    return {"metric": "fused rectified contraction TFLOP/s (4 rows blk r per launch)",
            "unit": "TFLOP/s", "dtype": "f32; bf16x3 split for the bf16x3 columns",
            "data": "synthetic",
            "config": {"workload": "kernel alone, A 250000 x r, B 2500 x r, N(0,1)"},
            "steps": steps, "warmup": warmup, "results": res}


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def cpu_baseline(p, frac=1):
    """fp64 oracle on the host over a bounded sample of the workload: the first W-step and the
    first H-step of sweep 0 at full size (about 15 s on 16 threads for the graph workload),
    each evaluated for every `frac`-th row of the factor it updates (the Gram solve and the
    block slicing run in full).  Scaled to one sweep of C W-steps and R H-steps: sweep time =
    frac * (C t_W + R t_H)."""
    import numpy as np
    from oracle import partition, salsa, schedule

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = os.cpu_count() or 1
    S = salsa.csr_matrix(p.m, p.n, p.row_ptr, p.col, p.val)
    ST = S.T.tocsr()
    st = salsa.State(p.W0, p.H0)
    rb = partition.bounds(p.m, p.block_m)
    cb = partition.bounds(p.n, p.block_n)
    R, C = len(rb) - 1, len(cb) - 1
    steps = schedule.sweep_schedule(p.seed, 0, R, C, True)
    kw = next(s for s in steps if s > 0) - 1
    kh = -next(s for s in steps if s < 0) - 1
    t0 = time.perf_counter()
    salsa.factor_step(S, st.A, st.B, cb[kw], cb[kw + 1], p.eta, p.momentum, st.VA,
                      rows=np.arange(0, p.m, frac))
    t1 = time.perf_counter()
    salsa.factor_step(ST, st.B, st.A, rb[kh], rb[kh + 1], p.eta, p.momentum, st.VB,
                      rows=np.arange(0, p.n, frac))
    t2 = time.perf_counter()
    sweep_s = frac * (C * (t1 - t0) + R * (t2 - t1))
    return {
        "value": 1.0 / sweep_s,
        "unit": "sweeps/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": (f"fp64 oracle at full size: first W-step ({t1 - t0:.1f} s) and first "
                   f"H-step ({t2 - t1:.1f} s) of sweep 0, "
                   + ("all rows" if frac == 1 else f"every {frac}th row")
                   + f"; sweep time = {frac} x ({C} W-steps + {R} H-steps)"),
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kernel-mb", action="store_true",
                    help="time the fused kernel alone at the shape of the paper's kernel table")
    ap.add_argument("--split-bf16", action="store_true",
                    help="opt-in variant at r_p = 16..512: both products of the dense kernel as "
                         "three bf16 MFMA products of two-term splits (fp32 stays the default)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="first run one plain 1 GiB copy kernel (calibrates rocprofv3 byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2608_21607_amd as nmd
    from workloads import gen

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.kernel_mb:
        print(json.dumps(kernel_mb(max(args.steps, 20), max(args.warmup, 2))), flush=True)
        return
    if args.copy_probe:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")  # 1 GiB
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)  # reads 1 GiB, writes 1 GiB
        torch.cuda.synchronize()
        log("copy probe: 1 GiB read + 1 GiB written by one elementwise kernel")
        del src, dst
    t0 = time.perf_counter()
    p = gen.config(args.config)
    log(f"workload {p.name}: m={p.m} n={p.n} r={p.r} nnz={p.nnz} "
        f"({time.perf_counter() - t0:.1f} s to generate)")

    ctx = nmd.Context(p.m, p.n, p.r, p.block_m, p.block_n, seed=p.seed, mode=p.mode,
                      eta=p.eta, momentum=p.momentum,
                      flags=nmd.FLAG_TIMING | (nmd.FLAG_SPLIT_BF16 if args.split_bf16 else 0))
    t0 = time.perf_counter()
    ctx.set_sparse_csr(p.row_ptr, p.col, p.val)
    log(f"ingest {time.perf_counter() - t0:.1f} s")
    W = torch.from_numpy(p.W0).cuda()
    H = torch.from_numpy(p.H0).cuda()
    torch.cuda.synchronize()

    f0 = ctx.objective(W, H)
    for k in range(args.warmup):
        ctx.sweep(W, H, 1)
        log(f"warmup sweep {k + 1}/{args.warmup} done")
    torch.cuda.synchronize()
    for kern in range(5):
        ctx.kernel_timing(kern, reset=True)
    ctx.dense_blocks(reset=True)

    stream = torch.cuda.current_stream()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for k in range(args.steps):
        ctx.sweep(W, H, 1)
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop)
    log(f"timed {args.steps} sweeps: {ms:.1f} ms")
    m1 = ctx.metrics(W, H)
    f1 = m1["objective"]
    assert np.isfinite(f1)

    # The objective after every sweep of the run above (warm-up and timed), from a second run of
    # the same sweeps from the same start with the per-sweep objective switched on, outside the
    # timed region.  The kernels are deterministic, so it is the same trajectory: its final
    # factors must equal the timed run's bit for bit.
    tctx = nmd.Context(p.m, p.n, p.r, p.block_m, p.block_n, seed=p.seed, mode=p.mode,
                       eta=p.eta, momentum=p.momentum,
                       flags=nmd.FLAG_SWEEP_OBJECTIVE
                       | (nmd.FLAG_SPLIT_BF16 if args.split_bf16 else 0))
    tctx.set_sparse_csr(p.row_ptr, p.col, p.val)
    W2 = torch.from_numpy(p.W0).cuda()
    H2 = torch.from_numpy(p.H0).cuda()
    tctx.sweep(W2, H2, args.warmup + args.steps)
    traj = [float(x) for x in tctx.sweep_objectives()]
    assert torch.equal(W2, W) and torch.equal(H2, H), "trajectory run differs from the timed run"
    tctx.close()
    del W2, H2
    rises = sum(1 for a, b in zip(traj, traj[1:]) if b > a)
    log(f"objective per sweep: {' '.join(f'{x:.4f}' for x in traj)} ({rises} rises)")

    rp = ((p.r + 15) // 16) * 16 if p.r <= 64 else ((p.r + 63) // 64) * 64  # padded rank
    kt = [ctx.kernel_timing(k) for k in range(5)]
    dense, sparse, factor, apply_, join = kt
    sweeps_per_s = args.steps / (ms / 1e3)
    dense_equiv = 4.0 * p.m * p.n * p.r * sweeps_per_s / 1e12
    dense_equiv_8mnr = 8.0 * p.m * p.n * p.r * sweeps_per_s / 1e12
    # The second product of the dense kernel runs its own MFMAs only for the 16 x 4 slices of
    # max(0, L) with a positive entry, or (r_p = 256, 512) per quad-column holding one,
    # counting the positive entries (2 r useful flops each).  Its algorithmic flops are the
    # first product's times the fraction of slices run whole plus 2 r per counted entry.
    g2_run, g2_total, g2_entries = ctx.dense_blocks()
    g2_frac = g2_run / g2_total if g2_total else 1.0
    split = args.split_bf16 and rp in (16, 32, 64, 128, 256, 512)
    # Executed-work rate: the first product plus the second product's live slices (the fp32
    # kernel's whole slices; every 16 x 4 slice of a live 16 x 32 tile for the split kernels).
    live_flops = dense["flops"] * (0.5 + 0.5 * g2_frac)
    if split and rp >= 256:
        # the method's own work: the first product plus 2 r per positive entry of max(0, L),
        # which the split kernels at r_p = 256 and 512 count (here g2_entries)
        dense_alg_flops = dense["flops"] * 0.5 + 2.0 * p.r * g2_entries
    elif split:
        dense_alg_flops = live_flops  # r_p <= 128: no entry count, the live-tile work
    else:
        dense_alg_flops = live_flops + 2.0 * p.r * g2_entries
    dense_s = dense["ms"] / 1e3
    dense_tflops = dense_alg_flops / dense_s / 1e12 if dense_s > 0 else 0.0
    dense_equiv_kernel = dense["flops"] / dense_s / 1e12 if dense_s > 0 else 0.0
    sparse_gbs = sparse["bytes"] / (sparse["ms"] / 1e3) / 1e9 if sparse["ms"] > 0 else 0.0
    # The split option runs both products as three bf16 products each: every algorithmic flop
    # costs three bf16 flops, so its roofline peak is a third of the bf16 MFMA peak.
    peak = PEAK_BF16_MFMA / 3.0 if split else PEAK_FP32_MFMA

    out = {
        "metric": METRIC,
        "value": sweeps_per_s,
        "unit": "sweeps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16x3 split / f32" if split else "f32",
        "data": "synthetic",
        "config": {
            "workload": p.name + {
                4: " (synthetic stand-in for the paper's connectome matrix)",
                5: " (synthetic stand-in for the paper's bigram-count matrix)",
            }.get(args.config, " (synthetic)"),
            "m": p.m, "n": p.n, "r": p.r, "nnz": p.nnz,
            "block_m": p.block_m, "block_n": p.block_n,
            "mode": p.mode, "eta": p.eta, "momentum": p.momentum, "seed": p.seed,
        },
        "dense_equiv_tflops": dense_equiv,
        "dense_equiv_frac_of_fp32_peak": dense_equiv / PEAK_FP32_MFMA,
        # the same dense-equivalent count for both halves of a sweep (W- and H-steps, 8 m n r);
        # the kernel skips most of that work, so this rate can exceed the peak
        "dense_equiv_8mnr_tflops": dense_equiv_8mnr,
        "dense_equiv_8mnr_frac_of_fp32_peak": dense_equiv_8mnr / PEAK_FP32_MFMA,
        # the sparse correction's algorithmic bytes over its own time; at r_p >= 320 it runs
        # beside the dense kernel (off the critical path), so that time is the one it takes there
        "sparse_pass_gbs": sparse_gbs,
        "sparse_pass_frac_of_hbm": sparse_gbs / PEAK_HBM,
        "sparse_beside_dense": rp >= 320 and not split,
        "kernel_ms_per_sweep": {
            "dense": dense["ms"] / args.steps, "sparse": sparse["ms"] / args.steps,
            "gram_inverse": factor["ms"] / args.steps, "solve_apply": apply_["ms"] / args.steps,
            # span of the side stream's Gram and inverse work (beside the dense kernel), and the
            # part of it the updates waited for
            "side_stream_wait": join["ms"] / args.steps,
        },
        "objective_before_after": [f0, f1],
        "objective_per_sweep": traj,
        "objective_rises": rises,
        "rmse_wjd_after": [m1["rmse"], m1["wjd"]],
        "roofline": {
            "bound": "mfma",
            "achieved": dense_tflops,
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": dense_tflops / peak,
            "traffic": measured_traffic(args.config, "split_bf16" if split else "fp32"),
            "kernel": ((f"bxl_kernel<{rp}>" if rp >= 256 else f"bx32_kernel<{rp}>")
                       if split else f"dense_kernel<{rp}>"),
            "launches": dense["launches"],
            "avg_launch_ms": dense["ms"] / max(1, dense["launches"]),
            "flops_per_launch": dense_alg_flops / max(1, dense["launches"]),
            "second_product_fraction_run": g2_frac,
            ("positive_entries_per_launch" if split else
             "second_product_positive_entries_per_launch"): g2_entries / max(1, dense["launches"]),
            "live_tile_rate_tflops": live_flops / dense_s / 1e12 if dense_s > 0 else 0.0,
            "dense_equiv_kernel_tflops": dense_equiv_kernel,
        },
    }
    if not args.no_cpu_baseline:
        log("timing the fp64 oracle on the host (bounded sample)")
        out["cpu_baseline"] = cpu_baseline(p)
    ctx.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
