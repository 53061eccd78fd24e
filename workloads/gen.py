"""Seeded generators for the five benchmark workloads and for small odd-shaped test problems.

Conventions (all generators):
  * RNG: numpy.random.Generator(PCG64(seed)).
  * S is returned in CSR form: row_ptr int64[m+1], col int32[nnz] (strictly increasing inside a
    row), val float32[nnz] (> 0).
  * Factors are float32: W is m x r row-major, H is r x n row-major, so L = W @ H.

The workloads stand in for the paper's datasets (Table of datasets, Sec. 2.5): they are not
reproductions of them.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np


@dataclass
class Problem:
    name: str
    m: int
    n: int
    r: int
    row_ptr: np.ndarray
    col: np.ndarray
    val: np.ndarray
    W0: np.ndarray
    H0: np.ndarray
    block_m: int
    block_n: int
    mode: str = "deterministic"  # or "stochastic"
    eta: float = 1.0
    momentum: float = 0.0
    seed: int = 1
    sweeps: int = 1
    meta: dict = field(default_factory=dict)

    @property
    def nnz(self) -> int:
        return int(self.row_ptr[-1])

    def coo(self):
        rows = np.repeat(np.arange(self.m, dtype=np.int64), np.diff(self.row_ptr))
        return rows, self.col.astype(np.int64), self.val


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def csr_from_keys(m: int, n: int, keys: np.ndarray, vals: np.ndarray):
    """CSR arrays from unique flat keys i*n + j (any order) and matching values."""
    order = np.argsort(keys, kind="stable")
    keys = keys[order]
    vals = vals[order]
    rows = keys // n
    cols = (keys - rows * n).astype(np.int32)
    counts = np.bincount(rows, minlength=m).astype(np.int64)
    row_ptr = np.zeros(m + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    return row_ptr, cols, np.ascontiguousarray(vals, dtype=np.float32)


# --------------------------------------------------------------------------------------------
# Initial factors
# --------------------------------------------------------------------------------------------

def sign_constrained_init(m: int, n: int, r: int, mean_s: float, seed: int):
    """A > 0 and B < 0, so that max(0, W H) is all zero at the start (Sec. 4.3, origins of
    sparsity).  The scale s makes E[L_ij] = -mean_s: with g ~ |N(0,1)|, E[g]^2 = 2/pi, so
    E[L_ij] = -s^2 r (2/pi), and s^2 = (pi/2) mean_s / r."""
    g = _rng(seed)
    s = math.sqrt((math.pi / 2.0) * float(mean_s) / r)
    W = (s * np.abs(g.standard_normal((m, r)))).astype(np.float32)
    H = (-s * np.abs(g.standard_normal((r, n)))).astype(np.float32)
    return W, H


def gaussian_init(m: int, n: int, r: int, std: float, seed: int):
    g = _rng(seed)
    W = (std * g.standard_normal((m, r))).astype(np.float32)
    H = (std * g.standard_normal((r, n))).astype(np.float32)
    return W, H


# --------------------------------------------------------------------------------------------
# Planted problems: S = max(0, W0 H0 - tau) with tau fixing the number of positive entries
# --------------------------------------------------------------------------------------------

def _top_k_threshold(W0: np.ndarray, H0: np.ndarray, k: int, seed: int, chunk_rows: int,
                     direct_limit: int = 40_000_000):
    """Exact selection of the k largest entries of L0 = W0 H0 (fp64 products of the fp32
    factors), returned as (flat keys, values, tau) where tau is the (k+1)-th largest value."""
    m, n = W0.shape[0], H0.shape[1]
    W = W0.astype(np.float64)
    H = H0.astype(np.float64)
    total = m * n
    if total <= direct_limit:
        flat = (W @ H).ravel()
        idx = np.argpartition(flat, total - k - 1)
        tau = flat[idx[total - k - 1]]
        top = idx[total - k:]
        return top.astype(np.int64), flat[top], float(tau)
    # Two passes: a sampled quantile gives a safe lower bound, then exact selection among the
    # candidates above it.
    g = _rng(seed ^ 0x5EED)
    ns = 2_000_000
    si = g.integers(0, m, ns)
    sj = g.integers(0, n, ns)
    sv = np.einsum("ij,ji->i", W[si], H[:, sj])
    frac = k / total
    q = max(0.0, 1.0 - 1.3 * frac - 5.0 * math.sqrt(frac / ns))
    lo = float(np.quantile(sv, q))
    while True:
        keys, vals = [], []
        for r0 in range(0, m, chunk_rows):
            blk = W[r0:r0 + chunk_rows] @ H
            ii, jj = np.nonzero(blk > lo)
            keys.append((ii.astype(np.int64) + r0) * n + jj)
            vals.append(blk[ii, jj])
        keys = np.concatenate(keys)
        vals = np.concatenate(vals)
        if keys.size >= k + 1:
            break
        lo -= 1.0 + abs(lo)
    c = keys.size
    idx = np.argpartition(vals, c - k - 1)
    tau = vals[idx[c - k - 1]]
    top = idx[c - k:]
    return keys[top], vals[top], float(tau)


def planted(m: int, n: int, d: int, density: float, seed: int, chunk_rows: int = 2048):
    """Planted problem: W0 (m x d), H0 (d x n) ~ N(0,1) fp32, L0 = W0 H0, tau chosen so that
    exactly floor(density*m*n) entries of L0 exceed it, S = max(0, L0 - tau)."""
    g = _rng(seed)
    W0 = g.standard_normal((m, d)).astype(np.float32)
    H0 = g.standard_normal((d, n)).astype(np.float32)
    k = int(math.floor(density * m * n))
    keys, vals, tau = _top_k_threshold(W0, H0, k, seed, chunk_rows)
    v = (vals - tau).astype(np.float32)
    keep = v > 0
    row_ptr, col, val = csr_from_keys(m, n, keys[keep], v[keep])
    return row_ptr, col, val, {"tau": tau, "k": k, "W_planted": W0, "H_planted": H0}


# --------------------------------------------------------------------------------------------
# Identity matrix and its exact rank-3 completion (Corollary 1, eq. Omega)
# --------------------------------------------------------------------------------------------

def identity(n: int):
    row_ptr = np.arange(n + 1, dtype=np.int64)
    col = np.arange(n, dtype=np.int32)
    val = np.ones(n, dtype=np.float32)
    return row_ptr, col, val


def identity_exact_factors(n: int, dtype=np.float64):
    """Rows [cos t_i, sin t_i, 1] and columns [cos t_j, sin t_j, -c]/(1-c), t_k = 2 pi k / n,
    c = cos(2 pi / n); their product is the matrix Omega of Corollary 1 (eq. Omega)."""
    t = 2.0 * np.pi * np.arange(n) / n
    c = math.cos(2.0 * math.pi / n)
    W = np.stack([np.cos(t), np.sin(t), np.ones(n)], axis=1)
    H = np.stack([np.cos(t), np.sin(t), -c * np.ones(n)], axis=0) / (1.0 - c)
    return W.astype(dtype), H.astype(dtype)


# --------------------------------------------------------------------------------------------
# Graph-like power-law count matrix (stand-in for a connectome)
# --------------------------------------------------------------------------------------------

def graph_powerlaw(n: int, nnz_target: int, seed: int, alpha: float = 2.2,
                   communities: int = 50, comm_frac: float = 0.3,
                   mu: float = 0.7, sigma: float = 1.0, cap_frac: float = 0.1):
    """Directed Chung-Lu sampler with power-law expected degrees.

    Out- and in-weights are Pareto(alpha) with minimum 1, rescaled to the target mean degree
    and capped at cap_frac*n.  A fraction comm_frac of the draws stays inside one of
    `communities` planted communities (uniform node assignment; a community is drawn in
    proportion to its out-weight mass); the rest is global, i proportional to w_out and j to
    w_in.  Draws are deduplicated until nnz_target unique pairs remain, then every empty row
    and column receives one entry.  Values are counts round(LogNormal(mu, sigma)), redrawn
    while 0.  Node ids are finally permuted at random (one permutation for rows and columns).
    """
    g = _rng(seed)
    mean_deg = nnz_target / n

    def weights():
        w = (1.0 - g.random(n)) ** (-1.0 / (alpha - 1.0))  # Pareto(alpha), x_min = 1
        w = w * (mean_deg / w.mean())
        return np.minimum(w, cap_frac * n)

    w_out = weights()
    w_in = weights()
    comm = g.integers(0, communities, n)
    members = [np.nonzero(comm == c)[0] for c in range(communities)]
    cdf_out = np.cumsum(w_out) / w_out.sum()
    cdf_in = np.cumsum(w_in) / w_in.sum()
    comm_mass = np.array([w_out[mb].sum() for mb in members])
    comm_cdf = np.cumsum(comm_mass) / comm_mass.sum()
    m_cdf_out = [np.cumsum(w_out[mb]) / w_out[mb].sum() for mb in members]
    m_cdf_in = [np.cumsum(w_in[mb]) / w_in[mb].sum() for mb in members]

    def draw(count):
        n_comm = int(round(count * comm_frac))
        n_glob = count - n_comm
        i_g = np.searchsorted(cdf_out, g.random(n_glob), side="right")
        j_g = np.searchsorted(cdf_in, g.random(n_glob), side="right")
        cs = np.searchsorted(comm_cdf, g.random(n_comm), side="right")
        i_c = np.empty(n_comm, dtype=np.int64)
        j_c = np.empty(n_comm, dtype=np.int64)
        for c in range(communities):
            sel = np.nonzero(cs == c)[0]
            if sel.size == 0:
                continue
            mb = members[c]
            i_c[sel] = mb[np.searchsorted(m_cdf_out[c], g.random(sel.size), side="right")]
            j_c[sel] = mb[np.searchsorted(m_cdf_in[c], g.random(sel.size), side="right")]
        i = np.minimum(np.concatenate([i_g, i_c]), n - 1)
        j = np.minimum(np.concatenate([j_g, j_c]), n - 1)
        return i.astype(np.int64) * n + j

    keys = np.unique(draw(int(nnz_target * 1.35)))
    while keys.size < nnz_target:
        keys = np.unique(np.concatenate([keys, draw(int((nnz_target - keys.size) * 1.6) + 1000)]))
    if keys.size > nnz_target:
        keys = np.sort(g.choice(keys, nnz_target, replace=False))
    rows = keys // n
    cols = keys % n
    # at least one entry in every row and every column
    extra = []
    empty_r = np.setdiff1d(np.arange(n), np.unique(rows))
    if empty_r.size:
        extra.append(empty_r * n + np.searchsorted(cdf_in, g.random(empty_r.size), side="right").clip(0, n - 1))
    empty_c = np.setdiff1d(np.arange(n), np.unique(cols))
    if empty_c.size:
        extra.append(np.searchsorted(cdf_out, g.random(empty_c.size), side="right").clip(0, n - 1) * n + empty_c)
    if extra:
        keys = np.unique(np.concatenate([keys] + extra))
    # values: zero-truncated rounded lognormal counts
    vals = np.rint(g.lognormal(mu, sigma, keys.size))
    zero = vals == 0
    while zero.any():
        vals[zero] = np.rint(g.lognormal(mu, sigma, int(zero.sum())))
        zero = vals == 0
    # relabel nodes
    perm = g.permutation(n)
    rows = perm[keys // n]
    cols = perm[keys % n]
    row_ptr, col, val = csr_from_keys(n, n, rows * n + cols, vals.astype(np.float32))
    return row_ptr, col, val


# --------------------------------------------------------------------------------------------
# Rectangular Zipf co-occurrence matrix (stand-in for bigram counts)
# --------------------------------------------------------------------------------------------

def _zipf_probs(k: int, s: float):
    p = np.arange(1, k + 1, dtype=np.float64) ** (-s)
    return p / p.sum()


def cooccurrence_zipf(m: int, n: int, nnz_target: int, seed: int, s: float = 1.1,
                      lam: float = 3.0):
    """Pairs (i, j) drawn N times with probability p_i q_j, p and q Zipf(s) in index order
    (a frequency-sorted vocabulary), deduplicated.  N is chosen so that the expected number of
    distinct pairs is nnz_target.  Each row receives Poisson(N p_i) draws; rows with many draws
    are sampled column by column with the exact presence probability 1 - (1 - q_j)^K, the
    others by drawing K columns and deduplicating.  Values are log(1 + c), c ~ Poisson(lam)
    redrawn while 0."""
    g = _rng(seed)
    p = _zipf_probs(m, s)
    q = _zipf_probs(n, s)
    lq = np.log1p(-q)

    # expected distinct pairs for N draws: sum_i sum_j 1 - exp(-N p_i q_j)
    xs = np.geomspace(1e-3, 1e9, 400)
    fx = np.array([np.sum(-np.expm1(-x * q)) for x in xs])

    def expected(N):
        return np.sum(np.interp(np.log(N * p), np.log(xs), fx))

    lo, hi = 1.0, 1e12
    for _ in range(100):
        mid = math.sqrt(lo * hi)
        if expected(mid) < nnz_target:
            lo = mid
        else:
            hi = mid
    N = math.sqrt(lo * hi)
    K = g.poisson(N * p)
    cdf_q = np.cumsum(q)
    heavy = K > n // 4
    rows_out, cols_out = [], []
    for i in np.nonzero(heavy)[0]:
        pres = g.random(n) < -np.expm1(K[i] * lq)
        js = np.nonzero(pres)[0]
        rows_out.append(np.full(js.size, i, dtype=np.int64))
        cols_out.append(js.astype(np.int64))
    light = np.nonzero(~heavy & (K > 0))[0]
    # light rows in batches of about 5e7 draws
    start = 0
    csum = np.cumsum(K[light])
    while start < light.size:
        base = csum[start - 1] if start > 0 else 0
        stop = int(np.searchsorted(csum, base + 50_000_000, side="right"))
        stop = max(stop, start + 1)
        rs = light[start:stop]
        rr = np.repeat(rs.astype(np.int64), K[rs])
        cc = np.minimum(np.searchsorted(cdf_q, g.random(rr.size), side="right"), n - 1)
        keys = np.unique(rr * n + cc)
        rows_out.append(keys // n)
        cols_out.append(keys % n)
        start = stop
    rows = np.concatenate(rows_out)
    cols = np.concatenate(cols_out)
    c = g.poisson(lam, rows.size)
    zero = c == 0
    while zero.any():
        c[zero] = g.poisson(lam, int(zero.sum()))
        zero = c == 0
    vals = np.log1p(c.astype(np.float64)).astype(np.float32)
    row_ptr, col, val = csr_from_keys(m, n, rows * n + cols, vals)
    return row_ptr, col, val, {"draws": N}


# --------------------------------------------------------------------------------------------
# Small random problems for odd shapes and edge cases
# --------------------------------------------------------------------------------------------

def random_sparse(m: int, n: int, density: float, seed: int, empty_rows: int = 0,
                  empty_cols: int = 0, heavy_row_frac: float = 0.0, lo: float = 0.1,
                  hi: float = 2.0):
    """Uniformly placed nonzeros with values in [lo, hi).  Optionally the last `empty_rows`
    rows and `empty_cols` columns are left empty, and row 0 receives a share heavy_row_frac of
    all nonzeros."""
    g = _rng(seed)
    mm = max(1, m - empty_rows)
    nn = max(1, n - empty_cols)
    k = max(1, int(round(density * mm * nn)))
    keys = np.unique(g.integers(0, mm, k).astype(np.int64) * n + g.integers(0, nn, k))
    if heavy_row_frac > 0:
        kh = min(nn, int(heavy_row_frac * keys.size / max(1e-9, 1 - heavy_row_frac)))
        heavy = g.choice(nn, kh, replace=False).astype(np.int64)
        keys = np.unique(np.concatenate([keys, heavy]))
    vals = g.uniform(lo, hi, keys.size).astype(np.float32)
    return csr_from_keys(m, n, keys, vals)


# --------------------------------------------------------------------------------------------
# The five workloads
# --------------------------------------------------------------------------------------------

CONFIGS = {
    1: dict(name="planted r=8, 1000x1000", m=1000, n=1000, r=8, block_m=256, block_n=256,
            mode="deterministic", eta=1.0, momentum=0.0, sweeps=3),
    2: dict(name="identity r=3, 4096x4096", m=4096, n=4096, r=3, block_m=1024, block_n=1024,
            mode="deterministic", eta=1.0, momentum=0.0, sweeps=200),
    3: dict(name="planted r=64, 32768x32768", m=32768, n=32768, r=64, block_m=4096,
            block_n=4096, mode="stochastic", eta=1.0, momentum=0.9, sweeps=5),
    # Both sparse count matrices take the step size 0.1, the value the paper's hyperparameter
    # table (appendix on experimental settings) uses where its default of 1 is too large (its
    # bigram models at ranks 16 to 512).  At 1 (momentum 0.9) the graph stand-in's objective
    # falls for about 20 sweeps and then diverges, and the co-occurrence stand-in's within a few.
    4: dict(name="graph r=256, 139255x139255, ~16.8M nnz", m=139255, n=139255, r=256,
            block_m=8192, block_n=8192, mode="stochastic", eta=0.1, momentum=0.9, sweeps=1),
    5: dict(name="co-occurrence r=512, 500000x50000, ~100M nnz", m=500000, n=50000, r=512,
            block_m=16384, block_n=8192, mode="stochastic", eta=0.1, momentum=0.9, sweeps=1),
}


def config(k: int, scale: float = 1.0) -> Problem:
    """Workload k (1..5).  scale < 1 shrinks m and n (and nnz proportionally to m*n for the
    planted and identity problems, to m for the sparse count matrices) for quick tests; the
    rank, block sizes and hyperparameters stay as in the full workload unless they no longer
    fit."""
    c = dict(CONFIGS[k])
    m = max(1, int(round(c["m"] * scale)))
    n = max(1, int(round(c["n"] * scale)))
    r = c["r"]
    data_seed = k
    init_seed = k + 1000
    meta = {}
    if k == 1:
        row_ptr, col, val, meta = planted(m, n, 8, 0.05, data_seed)
        W0, H0 = sign_constrained_init(m, n, r, float(val.mean()), init_seed)
    elif k == 2:
        row_ptr, col, val = identity(n)
        m = n
        W0, H0 = gaussian_init(m, n, r, 0.1, init_seed)
    elif k == 3:
        row_ptr, col, val, meta = planted(m, n, 64, 0.01, data_seed)
        W0, H0 = sign_constrained_init(m, n, r, float(val.mean()), init_seed)
    elif k == 4:
        n = m
        row_ptr, col, val = graph_powerlaw(n, int(round(16_800_000 * scale)), data_seed)
        W0, H0 = sign_constrained_init(m, n, r, float(val.mean()), init_seed)
    elif k == 5:
        row_ptr, col, val, meta = cooccurrence_zipf(m, n, int(round(100_000_000 * scale)), data_seed)
        W0, H0 = sign_constrained_init(m, n, r, float(val.mean()), init_seed)
    else:
        raise ValueError(k)
    bm = min(c["block_m"], m)
    bn = min(c["block_n"], n)
    return Problem(name=c["name"], m=m, n=n, r=r, row_ptr=row_ptr, col=col, val=val, W0=W0,
                   H0=H0, block_m=bm, block_n=bn, mode=c["mode"], eta=c["eta"],
                   momentum=c["momentum"], seed=k, sweeps=c["sweeps"], meta=meta)
