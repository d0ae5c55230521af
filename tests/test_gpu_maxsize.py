"""GPU checks at the largest sizes the C ABI accepts (N up to 2^32 - 1).

The oracle's full sort is out of reach at 2^31 and more elements, so these
tests check properties that fix the exact top-k at any size, computed on
the GPU in chunks: with v the k-th returned key,
  * every returned value is the input's value at the returned index, bit
    for bit, and the indices are distinct and in range;
  * the output is sorted by key descending, ties by index ascending;
  * no element with a key above v is missing (their count equals the
    number of returned keys above v);
  * the returned elements with key v are the smallest indices holding v.
Inputs are seeded synthetic vectors generated on the GPU.
"""

import numpy as np
import pytest

import paper_2608_12573_amd as pk
from gpu_util import note, torch

pytestmark = pytest.mark.gpu

CHUNK = 1 << 28


def _keys(t):
    """Order-preserving integer keys (int64) of an fp32 or bf16 tensor."""
    th = torch()
    if t.dtype == th.float32:
        b = t.view(th.int32).to(th.int64) & 0xFFFFFFFF
        return th.where(b >= 0x80000000, 0xFFFFFFFF - b, b | 0x80000000)
    b = t.view(th.int16).to(th.int64) & 0xFFFF
    return th.where(b >= 0x8000, 0xFFFF - b, b | 0x8000)


def _check_exact(x, k, vals, idx, info):
    th = torch()
    rec = pk.read_info(info)[0]
    assert int(rec["n_valid"]) == k
    N = x.numel()
    assert idx.dtype == th.int64 and int(idx.min()) >= 0 and int(idx.max()) < N
    assert th.unique(idx).numel() == k
    # values are bit copies of the input at the indices
    assert th.equal(_keys(vals), _keys(x[idx]))
    kv = _keys(vals)
    # sorted: key descending, ties by index ascending
    assert bool((kv[:-1] >= kv[1:]).all())
    same = kv[:-1] == kv[1:]
    assert bool((idx[:-1][same] < idx[1:][same]).all())
    v = int(kv[-1])
    above_out = int((kv > v).sum())
    above_in, ties = 0, []
    need = k - above_out
    for s in range(0, N, CHUNK):
        kc = _keys(x[s:s + CHUNK])
        above_in += int((kc > v).sum())
        if len(ties) < need:
            ties.extend((th.nonzero(kc == v).flatten()[:need - len(ties)] + s).tolist())
    assert above_in == above_out, (above_in, above_out)
    assert idx[above_out:].tolist() == ties[:need]
    return rec


def _gen(seed):
    g = torch().Generator(device="cuda")
    g.manual_seed(seed)
    return g


@pytest.mark.parametrize("k", [64, 1000])
def test_f32_2p31_plus5_normal(k):
    th = torch()
    N = (1 << 31) + 5
    note(f"max size f32 normal N={N} k={k}")
    x = th.randn(N, generator=_gen(31), device="cuda", dtype=th.float32)
    vals, idx, info = pk.topk(x, k, seed=3)
    rec = _check_exact(x, k, vals, idx, info)
    assert int(rec["status"]) == 0
    del x


def test_f32_2p31_plus5_large_k():
    # the multi-block refinement with indices past 2^31
    th = torch()
    N = (1 << 31) + 5
    note(f"max size f32 normal N={N} k=20000")
    x = th.randn(N, generator=_gen(32), device="cuda", dtype=th.float32)
    vals, idx, info = pk.topk(x, 20000, seed=4)
    _check_exact(x, 20000, vals, idx, info)
    del x


def test_bf16_max_n_closed_form():
    # N = 2^32 - 1 bf16 zeros with ten ones at the very end: every element
    # survives, the buffer overflows and the exact fallback runs over the
    # whole input; the answer is the ten ones, then the smallest indices of
    # the zeros
    th = torch()
    N = (1 << 32) - 1
    k = 100
    note(f"max size bf16 N={N} k={k} closed form")
    x = th.zeros(N, device="cuda", dtype=th.bfloat16)
    x[N - 10:] = 1.0
    vals, idx, info = pk.topk(x, k)
    rec = pk.read_info(info)[0]
    assert int(rec["status"]) in (1, 2)  # a fallback, whatever the sample saw
    want = list(range(N - 10, N)) + list(range(90))
    assert idx.tolist() == want
    assert vals[:10].float().eq(1.0).all() and vals[10:].float().eq(0.0).all()
    del x


def test_bf16_max_n_relu():
    th = torch()
    N = (1 << 32) - 1
    note(f"max size bf16 relu normal N={N} k=4096")
    x = th.empty(N, device="cuda", dtype=th.bfloat16)
    g = _gen(33)
    for s in range(0, N, CHUNK):
        n = min(CHUNK, N - s)
        x[s:s + n] = th.randn(n, generator=g, device="cuda", dtype=th.float32).clamp_(min=0.0).to(th.bfloat16)
    vals, idx, info = pk.topk(x, 4096, seed=5)
    rec = _check_exact(x, 4096, vals, idx, info)
    assert int(rec["status"]) == 0
    del x
