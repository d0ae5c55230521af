"""O1: exact top-k, the plain definition.

Test infrastructure (see the package docstring).

Sec. 3 (problem setup): return the k largest entries of x and their indices.
Under the total order of oracle.keys (key descending, then index ascending)
that is the first k positions of a stable sort of the indices by key,
descending.  Values are bit copies of the inputs.
"""

import numpy as np

from .keys import keys_of


def order_all(bits, dtype):
    """All indices in the total order (stable sort by key descending)."""
    key = keys_of(bits, dtype)
    return np.argsort(-key, kind="stable")


def topk(bits, dtype, k):
    """(values as bit patterns, int64 indices) of the exact top-k."""
    bits = np.asarray(bits)
    idx = order_all(bits, dtype)[:k].astype(np.int64)
    return bits[idx], idx


def topk_rows(bits2d, dtype, k):
    """O1 applied to every row of a [B, D] array; indices are columns."""
    B = bits2d.shape[0]
    vals = np.empty((B, k), dtype=bits2d.dtype)
    idx = np.empty((B, k), dtype=np.int64)
    for r in range(B):
        vals[r], idx[r] = topk(bits2d[r], dtype, k)
    return vals, idx
