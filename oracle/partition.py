"""Balanced block partition of the rows (or columns) of S.

The paper only says that the blocks (row sets I for parallel updates, column mini-batches J
for stochastic updates) are gated by memory and that an epoch loops over the rows and columns
of S (Sec. 4.1 and Sec. 5.1); it fixes no rule.  Reading used here: K = ceil(size / block)
blocks, block k covering [floor(k*size/K), floor((k+1)*size/K)).  Every block is at most the
requested size and sizes differ by at most one, so no tiny tail block (with an ill-conditioned
Gram matrix) appears.
"""


def num_blocks(size: int, block: int) -> int:
    return -(-size // block)


def bounds(size: int, block: int):
    """Start offsets of the K blocks plus the end, as a list of K+1 ints."""
    K = num_blocks(size, block)
    return [(k * size) // K for k in range(K + 1)]
