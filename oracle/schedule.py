"""Seeded per-sweep block order, written from the published definitions of its parts.

The paper draws "a random mini-batch J of column indices" for each stochastic update and
combines row and column subsampling (Sec. 4.1, stochastic least squares and complementarity);
it does not say how W- and H-updates interleave within an epoch.  Reading used here:

  * Generator: SplitMix64 (Steele, Lea and Flood, OOPSLA 2014), state advanced by the golden
    gamma 0x9E3779B97F4A7C15, output mixed by the two published multiply-xorshift rounds.
    The stream of sweep t starts from seed XOR (t * gamma mod 2^64).
  * Bounded integers: Lemire's multiply-and-reject method (ACM TOMACS 2019): with x uniform in
    [0, 2^64) the product x*k splits into high and low words; the high word is the result
    unless the low word falls below (2^64 - k) mod k, in which case x is redrawn.
  * Shuffle: Fisher-Yates in Durstenfeld's order (i from k-1 down to 1, swap a[i] with a[j],
    j uniform in [0, i]).  The column-block order sigma is drawn first, then the row-block
    order pi, from the same stream.
  * Interleave: W-steps (column blocks) and H-steps (row blocks) are merged in proportion:
    the next W-step comes first whenever (2w+1) R <= (2h+1) C, where w and h count the steps
    already emitted, so that with R == C the two strictly alternate starting with W.

Encoding: +(k+1) is the W-step of column block k, -(k+1) the H-step of row block k.
Deterministic (full-batch) sweeps list +1..+C then -1..-R: the W half accumulates over every
column block before a single solve, then the H half over every row block.
"""

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15


class SplitMix64:
    def __init__(self, state: int):
        self.state = state & MASK64

    def next(self) -> int:
        self.state = (self.state + GAMMA) & MASK64
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
        return z ^ (z >> 31)


def bounded(rng: SplitMix64, k: int) -> int:
    """Uniform integer in [0, k) by Lemire's method."""
    x = rng.next()
    prod = x * k
    low = prod & MASK64
    if low < k:
        threshold = ((1 << 64) - k) % k
        while low < threshold:
            x = rng.next()
            prod = x * k
            low = prod & MASK64
    return prod >> 64


def shuffled(rng: SplitMix64, k: int):
    a = list(range(k))
    for i in range(k - 1, 0, -1):
        j = bounded(rng, i + 1)
        a[i], a[j] = a[j], a[i]
    return a


def interleave(sigma, pi):
    C, R = len(sigma), len(pi)
    out, w, h = [], 0, 0
    while w < C or h < R:
        if h == R or (w < C and (2 * w + 1) * R <= (2 * h + 1) * C):
            out.append(sigma[w] + 1)
            w += 1
        else:
            out.append(-(pi[h] + 1))
            h += 1
    return out


def sweep_schedule(seed: int, t: int, R: int, C: int, stochastic: bool = True):
    """Step list of sweep t (0-based) for R row blocks and C column blocks."""
    if not stochastic:
        return [k + 1 for k in range(C)] + [-(k + 1) for k in range(R)]
    rng = SplitMix64((seed ^ ((t * GAMMA) & MASK64)) & MASK64)
    sigma = shuffled(rng, C)
    pi = shuffled(rng, R)
    return interleave(sigma, pi)
