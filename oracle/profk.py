"""O2: Prof-K step by step on the CPU (Sec. 3, "The Prof-K Algorithm").

Test infrastructure (see the package docstring).

For one vector of N values under plan (S, t, M, k_req):
  1. Sampling: S indices drawn i.i.d. uniform over [0, N) from Philox
     (oracle.philox; with-replacement reading in oracle.plan).
  2. Threshold estimation: tau = the t-th largest sampled key, duplicates
     counted with multiplicity (rank 1 is the largest).
  3. Filtering: the survivors are every i with key_i >= tau; their number
     'count' is exact (counting continues past M).
     Lexicographic plans (plan.lexicographic) compare (key, -index) pairs
     instead: stage 2 takes the t-th largest sampled pair (tau, -i_tau), and
     i survives iff key_i > tau, or key_i = tau and i <= i_tau.  Pairs are
     all distinct, so count is exactly the rank of the threshold pair even
     when values repeat (a plateau at tau no longer overflows the buffer).
  4. Refinement: if count < k_req (insufficient recall) or count > M (buffer
     overflow) the result is the exact top-k of the whole input (O1).
     Otherwise it is the top-k of the survivors in the total order; in
     relaxed mode, when k_req <= count < k, all 'count' survivors are
     returned in order and the rest of the output is padding (index -1,
     value -inf), with n_valid = count.

Plans with mode DIRECT skip stages 1-3 and return O1 directly.
"""

from dataclasses import dataclass

import numpy as np

from . import exact
from .keys import keys_of
from .philox import sample_indices
from .plan import MODE_DIRECT

STATUS_FILTERED = 0
STATUS_UNDERFLOW = 1
STATUS_OVERFLOW = 2
STATUS_DIRECT = 3

NEG_INF_BITS = {"f32": np.uint32(0xFF800000), "bf16": np.uint16(0xFF80)}


@dataclass
class Result:
    vals: np.ndarray      # bit patterns, length k
    idx: np.ndarray       # int64, length k (-1 past n_valid)
    status: int
    tau_key: int          # -1 when no threshold was drawn (DIRECT)
    count: int            # -1 when no filtering ran (DIRECT)
    n_valid: int
    tau_idx: int = -1     # lexicographic plans: index of the threshold pair


def sample_keys(key, plan, seed, row=0):
    """Stage 1: keys of the S sampled elements."""
    return key[sample_indices(seed, row, plan.S, len(key))]


def threshold(skeys, t):
    """Stage 2: the t-th largest sampled key (1-based, with multiplicity)."""
    return int(np.sort(skeys)[::-1][t - 1])


def survivors(key, tau):
    """Stage 3: ascending indices i with key_i >= tau."""
    return np.flatnonzero(key >= tau)


def threshold_lex(skeys, sidx, t):
    """Stage 2, lexicographic: the t-th largest sampled pair (key, -index),
    with multiplicity; returns (tau, i_tau)."""
    order = np.lexsort((sidx, -skeys.astype(np.int64)))   # key descending, index ascending
    j = order[t - 1]
    return int(skeys[j]), int(sidx[j])


def survivors_lex(key, tau, tau_idx):
    """Stage 3, lexicographic: ascending i with (key_i, -i) >= (tau, -tau_idx)."""
    i = np.arange(key.size)
    return np.flatnonzero((key > tau) | ((key == tau) & (i <= tau_idx)))


def run(bits, dtype, k, plan, seed, row=0, tau_override=None, key=None):
    """Prof-K on one vector.  tau_override replaces stages 1-2 (used to force
    the failure paths); it is a key, or for a lexicographic plan a
    (key, index) pair.  key: keys_of(bits, dtype) when the caller already
    holds it (large inputs checked under several seeds)."""
    bits = np.asarray(bits)
    key = keys_of(bits, dtype) if key is None else key
    if plan.mode == MODE_DIRECT and tau_override is None:
        v, i = exact.topk(bits, dtype, k)
        return Result(v, i, STATUS_DIRECT, -1, -1, k)
    lex = bool(getattr(plan, "lexicographic", False))
    tau_idx = -1
    if tau_override is not None:
        if lex:
            tau, tau_idx = (int(v) for v in tau_override)
        else:
            tau = int(tau_override)
    elif lex:
        sidx = sample_indices(seed, row, plan.S, len(key))
        tau, tau_idx = threshold_lex(key[sidx], sidx, plan.t)
    else:
        tau = threshold(sample_keys(key, plan, seed, row), plan.t)
    surv = survivors_lex(key, tau, tau_idx) if lex else survivors(key, tau)
    count = int(surv.size)
    if count < plan.k_req or count > plan.M:
        v, i = exact.topk(bits, dtype, k)
        status = STATUS_UNDERFLOW if count < plan.k_req else STATUS_OVERFLOW
        return Result(v, i, status, tau, count, k, tau_idx)
    order = surv[np.argsort(-key[surv], kind="stable")]
    take = order[:k].astype(np.int64)
    n_valid = int(take.size)
    vals = np.full(k, NEG_INF_BITS[dtype], dtype=bits.dtype)
    idx = np.full(k, -1, dtype=np.int64)
    vals[:n_valid] = bits[take]
    idx[:n_valid] = take
    return Result(vals, idx, STATUS_FILTERED, tau, count, n_valid, tau_idx)


def run_rows(bits2d, dtype, k, row_plan, seed, rows=None):
    """Per-row Prof-K (Sec. 3: applied to each batch element).  Row r uses
    counter word 1 = r, so rows draw independent samples.  Returns a list of
    Result, one per requested row, with column indices."""
    rows = range(bits2d.shape[0]) if rows is None else rows
    return [run(bits2d[r], dtype, k, row_plan, seed, row=r) for r in rows]


def run_batchtopk(bits2d, dtype, k_row, flat_plan, seed, key=None):
    """BatchTopK (Sec. 5, BatchTopK SAEs): the [B, D] matrix is flattened to
    N = B*D and the K = B*k_row largest entries are selected globally.
    Indices are flat (row*D + col).  key: as in run, for the flat view."""
    B = bits2d.shape[0]
    return run(bits2d.reshape(-1), dtype, B * k_row, flat_plan, seed, row=0, key=key)
