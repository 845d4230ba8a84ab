"""Q / KV partition index lists of a GPU's tile.

Test infrastructure only (see the package docstring).  The library takes these
lists as inputs; the oracle derives them here so that the tiles used in tests
can be checked against the paper's own examples.
"""


def basic_tile(g, a, b):
    """Basic 2-D tiling (Section 3.2): with n = a*b GPUs the assignment matrix
    is cut into tiles of height a (Q) and width b (KV); GPU g gets tile row
    r = g // a and tile column c = g mod a, i.e. Q partitions ra .. (r+1)a-1 and
    KV partitions cb .. (c+1)b-1."""
    r, c = g // a, g % a
    return list(range(r * a, (r + 1) * a)), list(range(c * b, (c + 1) * b))


def kvr_tile(g, a, b):
    """KV Partition Rotation (Section 3.3): the same Q partitions, but the KV
    footprint of tile column c = g mod a becomes the strided set
    {c + t*a : 0 <= t < b}."""
    q, _ = basic_tile(g, a, b)
    c = g % a
    return q, [c + t * a for t in range(b)]
