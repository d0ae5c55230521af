"""Pins for oracle.philox: numpy's Philox bit generator (an independent
implementation of Philox4x64-10) and exact big-integer arithmetic."""

import numpy as np
import pytest

from oracle import philox

M64 = (1 << 64) - 1


@pytest.mark.parametrize("key,ctr", [
    ((0, 0), (0, 0, 0, 0)),
    ((123, 456), (7, 8, 9, 10)),
    ((0xFFFFFFFFFFFFFFFF, 1), (0xFFFFFFFFFFFFFFFE, 3, 0, 0)),
    ((0x9E3779B97F4A7C15, 0), (5, 4096, 0, 0)),
])
def test_philox_matches_numpy(key, ctr):
    # numpy's generator advances the counter before producing each block, so
    # its stream from counter c is our blocks c+1, c+2, ...
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                          counter=np.array(ctr, dtype=np.uint64))
    raw = bg.random_raw(4 * 6)
    c0 = np.array([(ctr[0] + 1 + b) & M64 for b in range(6)], dtype=np.uint64)
    carry = np.array([1 if ctr[0] + 1 + b > M64 else 0 for b in range(6)], dtype=np.uint64)
    mine = philox.philox4x64_10((c0, np.uint64(ctr[1]) + carry, ctr[2], ctr[3]), key)
    mine = np.stack(mine, axis=1).reshape(-1)
    assert np.array_equal(mine, raw)


def test_philox_counter_zero_known_answer():
    # Block at counter 0 with key 0; numpy reaches it from counter 2^64 - 1.
    bg = np.random.Philox(key=np.zeros(2, np.uint64),
                          counter=np.full(4, M64, dtype=np.uint64))
    raw = bg.random_raw(4)
    mine = np.array(philox.philox4x64_10((0, 0, 0, 0), (0, 0)), dtype=np.uint64)
    assert np.array_equal(mine, raw)


def test_mulhilo_matches_bigint():
    g = np.random.default_rng(1)
    a = g.integers(0, 2**64, 5000, dtype=np.uint64)
    b = g.integers(0, 2**64, 5000, dtype=np.uint64)
    a[:3] = [0, M64, M64]
    b[:3] = [M64, M64, 1]
    hi, lo = philox.mulhilo64(a, b)
    for x, y, h, l in zip(a.tolist(), b.tolist(), hi.tolist(), lo.tolist()):
        p = x * y
        assert h == p >> 64 and l == p & M64


def test_sample_word_layout():
    seed, row, S = 77, 5, 23
    w = philox.sample_words(seed, row, S)
    for j in range(S):
        blk = philox.philox4x64_10((j // 4, row, 0, 0), (seed, 0))
        assert int(w[j]) == int(blk[j % 4])


@pytest.mark.parametrize("N", [1, 2, 3, 1000, 2**20, 2**28, 2**32 - 1])
def test_index_map_exact(N):
    g = np.random.default_rng(N % 97)
    u = g.integers(0, 2**64, 2000, dtype=np.uint64)
    u[:2] = [0, M64]
    idx = philox.index_of_word(u, N)
    exp = [(int(x) * N) >> 64 for x in u.tolist()]
    assert idx.tolist() == exp
    assert idx.min() >= 0 and idx.max() < N


def test_sample_indices_uniform_chi_square():
    from scipy.stats import chisquare
    N = 1 << 16
    idx = philox.sample_indices(3, 0, 200_000, N)
    counts = np.bincount(idx // (N // 64), minlength=64)
    assert chisquare(counts).pvalue > 1e-4


def test_rows_draw_different_streams():
    a = philox.sample_indices(0, 0, 64, 1 << 20)
    b = philox.sample_indices(0, 1, 64, 1 << 20)
    c = philox.sample_indices(1, 0, 64, 1 << 20)
    assert not np.array_equal(a, b) and not np.array_equal(a, c)
