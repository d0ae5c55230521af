"""GPU parity of the exact fallback for k <= 4096 (Sec. 3, stage 4: when the
buffer under- or overflows, the exact top-k of the whole input), on inputs
that drive each of its steps: many chunks merged in two levels, tie classes
too large for on-chip memory inside one chunk (cut in index order) and
inside a merge (cut by an index select), unaligned bases and odd k.

Results are compared bit for bit with the oracle, and all-equal inputs also
with their closed form: indices 0..k-1.
"""

import numpy as np
import pytest

import paper_2608_12573_amd as pk
import workloads
from oracle import keys as okeys, profk as oprofk
from gpu_util import compare, gpu_bf16, gpu_f32, host_bits, note, oracle_plan_of, plan_from_lib

pytestmark = pytest.mark.gpu


def _run(bits, dtype, g, k, seed=0):
    p = pk.plan(bits.size, k)
    q = oracle_plan_of(p)
    note(f"fallback {dtype} N={bits.size} k={k} S={p.S} t={p.t} M={p.M} mode={p.mode}")
    vals, idx, info = pk.topk(g, k, seed=seed, p=p)
    ref = oprofk.run(bits, dtype, k, q, seed)
    return compare(vals, idx, info, ref, dtype), ref, vals, idx


@pytest.mark.parametrize("k", [1, 64, 999, 4096])
@pytest.mark.parametrize("offset", [0, 1])
def test_all_equal_f32(k, offset):
    # every element survives the filter, so the buffer overflows; every
    # chunk holds one tie class larger than on-chip memory, and at k = 4096
    # so does every merge
    N = (1 << 22) + 5
    x = np.full(N, 1.5, dtype=np.float32)
    rec, ref, vals, idx = _run(okeys.f32_bits(x), "f32", gpu_f32(x, offset), k)
    assert ref.status == oprofk.STATUS_OVERFLOW
    assert np.array_equal(idx.cpu().numpy(), np.arange(k))
    assert np.all(host_bits(vals) == np.float32(1.5).view(np.uint32))


@pytest.mark.parametrize("offset", [0, 3])
def test_all_equal_bf16(offset):
    N = (1 << 21) + 7
    b = np.full(N, 0x3FC0, dtype=np.uint16)  # bf16 1.5
    for k in (100, 4096):
        rec, ref, vals, idx = _run(b, "bf16", gpu_bf16(b, offset), k)
        assert np.array_equal(idx.cpu().numpy(), np.arange(k))


@pytest.mark.parametrize("k", [512, 4093])
def test_wide_plateau_overflow(k):
    # 5e5 equal values from rank 101 on: each chunk keeps a part of the
    # plateau, and the merges of 16 chunks cut a tie class larger than
    # on-chip memory
    x = workloads.plateau_f32(1 << 24, seed=21, first_rank=101, width=500_000)
    rec, ref, _, _ = _run(okeys.f32_bits(x), "f32", gpu_f32(x), k)
    assert ref.status == oprofk.STATUS_OVERFLOW


@pytest.mark.parametrize("k", [7, 1000, 4093])
def test_forced_underflow_large(k):
    # a threshold above every key leaves no survivor: the fallback runs on
    # 2^24 + 3 unaligned values (a head and a tail outside the vectors)
    N = (1 << 24) + 3
    x = workloads.normal_f32(N, seed=22)
    bits = okeys.f32_bits(x)
    key = okeys.keys_of(bits, "f32")
    p = pk.plan(N, k)
    q = plan_from_lib(p)
    tau = int(key.max()) + 1
    note(f"fallback forced underflow N={N} k={k} tau={tau:#x}")
    vals, idx, info = pk.topk_tau(gpu_f32(x, 2), k, tau, p)
    ref = oprofk.run(bits, "f32", k, q, 0, tau_override=tau)
    assert ref.status == oprofk.STATUS_UNDERFLOW
    compare(vals, idx, info, ref, "f32")


def test_zero_ties_across_chunks_bf16():
    # 1000 positive values among 2^20 - 1000 zeros: with k = 4096 the k-th
    # key is +0, a tie class spread over every chunk, cut in the merges
    N = 1 << 20
    g = np.random.default_rng(23)
    b = np.zeros(N, dtype=np.uint16)
    pos = g.choice(N, 1000, replace=False)
    b[pos] = workloads.f32_to_bf16_bits(g.random(1000, dtype=np.float32) + np.float32(0.5))
    p = pk.plan(N, 4096)
    q = plan_from_lib(p)
    tau = int(okeys.keys_of(b, "bf16").max()) + 1
    note("fallback bf16 zero ties")
    vals, idx, info = pk.topk_tau(gpu_bf16(b, 1), 4096, tau, p)
    ref = oprofk.run(b, "bf16", 4096, q, 0, tau_override=tau)
    assert ref.status == oprofk.STATUS_UNDERFLOW
    compare(vals, idx, info, ref, "bf16")
    gi = idx.cpu().numpy()
    assert np.array_equal(np.sort(gi[:1000]), np.sort(pos))
    zeros = np.setdiff1d(np.arange(N), pos)[:4096 - 1000]
    assert np.array_equal(gi[1000:], zeros)
