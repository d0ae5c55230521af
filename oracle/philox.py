"""Philox4x64-10 and the sample-index map used by Stage 1 (Sampling).

Test infrastructure (see the package docstring).

The paper draws S sample indices uniformly (Sec. 3, stage 1) and says
nothing about the generator.  Reading used here: draws are independent and
uniform over [0, N) (with replacement), produced by the counter-based
generator Philox4x64 with 10 rounds from Salmon, Moraes, Dror and Shaw,
"Parallel random numbers: as easy as 1, 2, 3" (SC'11):

  * state: four 64-bit counter words, key: two 64-bit words;
  * one round maps (x0, x1, x2, x3) with key (k0, k1) to
        (hi(B*x2) ^ x1 ^ k0,  lo(B*x2),  hi(A*x0) ^ x3 ^ k1,  lo(A*x0))
    where A = 0xD2E7470EE14C6C93, B = 0xCA5A826395121157 and hi/lo are the
    upper/lower halves of the 128-bit product;
  * between rounds the key is advanced by the Weyl constants
    (0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B); ten rounds in all.

Draw j of row r under seed s is output word (j mod 4) of the block with
counter (floor(j/4), r, 0, 0) and key (s, 0).  The index is the upper 64 bits
of the 128-bit product u * N, i.e. floor(u * N / 2**64), whose relative bias
is below N / 2**64.
"""

import numpy as np

_M32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)
_MUL_A = 0xD2E7470EE14C6C93
_MUL_B = 0xCA5A826395121157
_WEYL_0 = 0x9E3779B97F4A7C15
_WEYL_1 = 0xBB67AE8584CAA73B
_ROUNDS = 10


def _u64(v):
    return np.asarray(v, dtype=np.uint64)


def mulhilo64(a, b):
    """(hi, lo) 64-bit halves of the 128-bit product of uint64 arrays a, b,
    assembled from 32-bit partial products."""
    a = _u64(a)
    b = _u64(b)
    a0, a1 = a & _M32, a >> _S32
    b0, b1 = b & _M32, b >> _S32
    p00 = a0 * b0
    p01 = a0 * b1
    p10 = a1 * b0
    p11 = a1 * b1
    mid = (p00 >> _S32) + (p01 & _M32) + (p10 & _M32)
    hi = p11 + (p01 >> _S32) + (p10 >> _S32) + (mid >> _S32)
    lo = (p00 & _M32) | ((mid & _M32) << _S32)
    return hi, lo


def philox4x64_10(ctr, key):
    """Philox4x64-10 block function.

    ctr: four uint64 arrays (broadcastable), key: two uint64 arrays.
    Returns the four uint64 output words."""
    x0, x1, x2, x3 = (_u64(c) for c in ctr)
    k0, k1 = (_u64(k) for k in key)
    x0, x1, x2, x3 = np.broadcast_arrays(x0, x1, x2, x3)
    for r in range(_ROUNDS):
        if r > 0:
            k0 = k0 + _u64(_WEYL_0)
            k1 = k1 + _u64(_WEYL_1)
        hi_a, lo_a = mulhilo64(_u64(_MUL_A), x0)
        hi_b, lo_b = mulhilo64(_u64(_MUL_B), x2)
        x0, x1, x2, x3 = hi_b ^ x1 ^ k0, lo_b, hi_a ^ x3 ^ k1, lo_a
    return x0, x1, x2, x3


def sample_words(seed, row, S):
    """The S raw 64-bit draws of one row: draw j is word (j mod 4) of the
    block with counter (j // 4, row, 0, 0) and key (seed, 0)."""
    S = int(S)
    nblk = (S + 3) // 4
    blk = np.arange(nblk, dtype=np.uint64)
    out = philox4x64_10((blk, _u64(row), _u64(0), _u64(0)),
                        (_u64(seed), _u64(0)))
    words = np.stack(out, axis=1).reshape(-1)
    return words[:S]


def index_of_word(u, N):
    """floor(u * N / 2**64) for uint64 words u: a uniform index in [0, N)."""
    hi, _ = mulhilo64(_u64(u), _u64(N))
    return hi.astype(np.int64)


def sample_indices(seed, row, S, N):
    """The S sample indices of one row (Sec. 3, stage 1)."""
    return index_of_word(sample_words(seed, row, S), N)
