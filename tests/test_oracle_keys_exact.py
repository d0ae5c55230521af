"""Pins for the total order (oracle.keys) and O1 (oracle.exact).

Everything here is checked against something other than the oracle's own
formulas: numpy float comparisons, an exhaustive sweep of all bf16 patterns,
a brute-force comparator written on float semantics, numpy lexsort, and
torch.topk values.
"""

import functools
import math

import numpy as np
import pytest

from oracle import exact, keys
import workloads


def _float_rank_cmp(x):
    """Comparator on float semantics (no integer keys): +NaN above all,
    -NaN below all, -0.0 below +0.0, otherwise numeric; ties by index."""
    def cls(v):
        if math.isnan(v):
            return 2 if math.copysign(1.0, v) > 0 else -2
        return 0

    def cmp(i, j):
        a, b = float(x[i]), float(x[j])
        ca, cb = cls(a), cls(b)
        if ca != cb:
            return -1 if ca > cb else 1
        if ca == 0 and a != b:
            return -1 if a > b else 1
        if ca == 0 and a == 0.0 and b == 0.0:
            sa, sb = math.copysign(1.0, a), math.copysign(1.0, b)
            if sa != sb:
                return -1 if sa > sb else 1
        return -1 if i < j else (1 if i > j else 0)
    return cmp


def test_key_u32_orders_like_floats():
    g = np.random.default_rng(11)
    bits = g.integers(0, 2**32, 200_000, dtype=np.uint64).astype(np.uint32)
    f = bits.view(np.float32)
    finite = np.isfinite(f)
    bits, f = bits[finite], f[finite]
    a, b = f[:-1], f[1:]
    ka, kb = keys.key_u32(bits[:-1]), keys.key_u32(bits[1:])
    differ = a != b
    assert np.array_equal((ka < kb)[differ], (a < b)[differ])
    same = bits[:-1] == bits[1:]
    assert np.all((ka == kb) == same)


def test_key_u32_special_values_strictly_increasing():
    seq = [0xFFC00000, 0xFF800000, 0xBF800000, 0x80000001, 0x80000000,
           0x00000000, 0x00000001, 0x3F800000, 0x7F800000, 0x7FC00000]
    kk = keys.key_u32(np.array(seq, dtype=np.uint32)).astype(np.int64)
    assert np.all(np.diff(kk) > 0)


def test_key_u16_exhaustive_against_fp32_expansion():
    b16 = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    as_f32 = (b16.astype(np.uint32) << np.uint32(16)).view(np.float32)
    k16 = keys.key_u16(b16).astype(np.int64)
    order = np.argsort(k16)
    f_sorted = as_f32[order]
    fin = np.isfinite(f_sorted)
    fs = f_sorted[fin]
    assert np.all(fs[:-1] <= fs[1:])
    assert np.array_equal(k16, (keys.key_u32(b16.astype(np.uint32) << np.uint32(16)) >> np.uint32(16)).astype(np.int64))
    assert np.array_equal(keys.bits_from_key_u16(keys.key_u16(b16)), b16)
    assert len(np.unique(k16)) == 65536


def test_key_u32_inverse():
    g = np.random.default_rng(12)
    bits = g.integers(0, 2**32, 100_000, dtype=np.uint64).astype(np.uint32)
    assert np.array_equal(keys.bits_from_key_u32(keys.key_u32(bits)), bits)


@pytest.mark.parametrize("seed", range(30))
def test_o1_brute_force_comparator(seed):
    g = np.random.default_rng(seed)
    n = int(g.integers(1, 14))
    x = workloads.special_f32(n, seed=seed)
    expected = sorted(range(n), key=functools.cmp_to_key(_float_rank_cmp(x)))
    bits = keys.f32_bits(x)
    for k in range(1, n + 1):
        v, i = exact.topk(bits, "f32", k)
        assert list(i) == expected[:k]
        assert np.array_equal(v, bits[expected[:k]])


@pytest.mark.parametrize("seed", range(10))
def test_o1_bf16_brute_force(seed):
    g = np.random.default_rng(100 + seed)
    n = int(g.integers(1, 40))
    b = g.integers(0x3F00, 0x3F08, n).astype(np.uint16)
    b[g.random(n) < 0.2] = 0x8000
    b[g.random(n) < 0.2] = 0x0000
    x = (b.astype(np.uint32) << np.uint32(16)).view(np.float32)
    expected = sorted(range(n), key=functools.cmp_to_key(_float_rank_cmp(x)))
    k = int(g.integers(1, n + 1))
    v, i = exact.topk(b, "bf16", k)
    assert list(i) == expected[:k]


def test_o1_upper_set_property_random_ties():
    g = np.random.default_rng(7)
    x = g.integers(0, 50, 3000).astype(np.float32)
    bits = keys.f32_bits(x)
    for k in (1, 17, 999, 3000):
        _, idx = exact.topk(bits, "f32", k)
        sel = np.zeros(x.size, bool)
        sel[idx] = True
        # every selected element precedes every unselected one
        worst_sel_val = x[idx[-1]]
        assert np.all(x[~sel] <= worst_sel_val)
        tie_unsel = np.flatnonzero(~sel & (x == worst_sel_val))
        tie_sel = idx[x[idx] == worst_sel_val]
        if tie_unsel.size:
            assert tie_sel.max() < tie_unsel.min()
        # output order: value non-increasing, index ascending inside ties
        xv = x[idx]
        assert np.all(xv[:-1] >= xv[1:])
        same = xv[:-1] == xv[1:]
        assert np.all(idx[:-1][same] < idx[1:][same])


def test_o1_matches_lexsort():
    g = np.random.default_rng(8)
    x = g.standard_normal(50_000).astype(np.float32)
    x[g.random(x.size) < 0.3] = 0.25
    bits = keys.f32_bits(x)
    ref = np.lexsort((np.arange(x.size), -x.astype(np.float64)))
    for k in (1, 100, 20_000):
        _, idx = exact.topk(bits, "f32", k)
        assert np.array_equal(idx, ref[:k])


def test_o1_values_match_torch_topk_tie_free():
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(9)
    x = g.permutation(200_000).astype(np.float32) - 1e5
    bits = keys.f32_bits(x)
    for k in (1, 64, 5000):
        v, idx = exact.topk(bits, "f32", k)
        tv, ti = torch.topk(torch.from_numpy(x), k, sorted=True)
        assert np.array_equal(v.view(np.float32), tv.numpy())
        assert np.array_equal(idx, ti.numpy())


def test_o1_all_equal_gives_first_indices():
    bits = keys.f32_bits(np.full(1000, 3.5, np.float32))
    _, idx = exact.topk(bits, "f32", 77)
    assert np.array_equal(idx, np.arange(77))


def test_o1_ramp_closed_form():
    # float32(i) for i in [0, n): above 2^24 the spacing is 2, so runs of
    # equal values appear.  The expected order lists runs in descending
    # value, each in ascending index order.
    n = 2**24 + 4099
    x = workloads.ramp_f32(n)
    xv = x[2**24 - 10:]
    base = 2**24 - 10
    starts = np.flatnonzero(np.r_[True, xv[1:] != xv[:-1]])
    ends = np.r_[starts[1:], xv.size]
    runs = [np.arange(s, e) + base for s, e in zip(starts, ends)]
    expected = np.concatenate(runs[::-1])
    k = 3001
    _, idx = exact.topk(keys.f32_bits(x), "f32", k)
    assert np.array_equal(idx, expected[:k])
    assert not np.array_equal(idx, np.arange(n - 1, n - 1 - k, -1))


def test_o1_k_equals_n_is_a_full_sort():
    g = np.random.default_rng(10)
    x = workloads.special_f32(500, seed=3)
    bits = keys.f32_bits(x)
    _, idx = exact.topk(bits, "f32", 500)
    assert np.array_equal(np.sort(idx), np.arange(500))
    kk = keys.key_u32(bits[idx]).astype(np.int64)
    assert np.all(np.diff(kk) <= 0)
    same = np.diff(kk) == 0
    assert np.all(np.diff(idx)[same] > 0)
