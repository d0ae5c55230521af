"""GPU parity of the tie-exact (lexicographic) filter rule against the CPU
oracle: bit-exact results, and the same status, threshold key and survivor
count, on inputs where ties at the threshold are the rule rather than the
exception.  Count equality also pins the threshold pair's index, since the
count is that pair's exact rank."""

import dataclasses

import numpy as np
import pytest

import paper_2608_12573_amd as pk
import workloads
from oracle import keys as okeys, plan as oplan, profk as oprofk
from gpu_util import compare, gpu_bf16, gpu_f32, note, oracle_plan_of, torch
from test_gpu_rows import _check_rows

pytestmark = pytest.mark.gpu


def _flat(bits, dtype, k, seed, **kw):
    p = pk.plan(bits.size, k, 1e-6, 1.0, lexicographic=1, **kw)
    q = oracle_plan_of(p, lexicographic=1, **kw)
    note(f"lex flat {dtype} N={bits.size} k={k} seed={seed} S={p.S} t={p.t} M={p.M} mode={p.mode}")
    g = gpu_f32(bits.view(np.float32)) if dtype == "f32" else gpu_bf16(bits)
    vals, idx, info = pk.topk(g, k, seed=seed, p=p)
    ref = oprofk.run(bits, dtype, k, q, seed)
    compare(vals, idx, info, ref, dtype)
    return ref


def test_lex_plateau_stays_in_the_buffer():
    # half of the input sits on one value near the top: the key rule
    # overflows (every plateau element survives), the pair rule does not
    x = workloads.normal_f32(2**20 + 11, seed=12)
    x[np.random.default_rng(5).random(x.size) < 0.5] = 4.0
    bits = okeys.f32_bits(x)
    ref = _flat(bits, "f32", 64, seed=3)
    assert ref.status == oprofk.STATUS_FILTERED
    plain = oprofk.run(bits, "f32", 64, oracle_plan_of(pk.plan(x.size, 64)), 3)
    assert plain.status == oprofk.STATUS_OVERFLOW


def test_lex_constant_input_revisits_the_draws():
    # every draw ties at tau, more than the tied-index list holds
    bits = okeys.f32_bits(np.full(2**20, 1.5, dtype=np.float32))
    ref = _flat(bits, "f32", 100, seed=7)
    assert ref.status == oprofk.STATUS_FILTERED
    assert list(ref.idx) == list(range(100))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_lex_bf16_natural_ties(seed):
    # bf16 keeps 8 bits of mantissa: many elements equal the threshold
    bits = workloads.f32_to_bf16_bits(workloads.normal_f32(2**21 + 5, seed=40 + seed))
    ref = _flat(bits, "bf16", 16, seed)          # t <= 8: tau would be chosen in the filter
    assert ref.status == oprofk.STATUS_FILTERED


def test_lex_ramp_with_repeats_many_ties():
    x = (np.arange(2**20) // 4096).astype(np.float32)   # runs of 4096 equal values
    ref = _flat(okeys.f32_bits(x), "f32", 1000, seed=5)
    assert ref.status == oprofk.STATUS_FILTERED


def test_lex_big_k_with_ties():
    x = np.round(workloads.normal_f32(2**21 + 3, seed=22) * 8).astype(np.float32)
    ref = _flat(okeys.f32_bits(x), "f32", 20000, seed=1)
    assert ref.status == oprofk.STATUS_FILTERED


def test_lex_tiny_sample():
    # 64 draws (t = 3): a loose threshold and a large buffer
    x = workloads.normal_f32(2**20, seed=2)
    ref = _flat(okeys.f32_bits(x), "f32", 64, seed=0, S_min=64, S_max=64,
                force_mode=pk.FORCE_FILTER, eps_split=0.999999)
    assert ref.status == oprofk.STATUS_FILTERED


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_lex_rows(dtype):
    B, D, k = 48, 8192, 16
    bits = workloads.relu_normal_bf16((B, D), seed=9) if dtype == "bf16" else \
        okeys.f32_bits(np.round(workloads.normal_f32(B * D, seed=9) * 16).astype(np.float32)).reshape(B, D)
    p = pk.plan_rows(D, k, 1e-6, 1.0, lexicographic=1)
    q = oplan.plan_rows(D, k, 1e-6, 1.0, dataclasses.replace(oplan.ROW_OPTS, lexicographic=True))
    assert (q.S, q.t, q.M) == (p.S, p.t, p.M) and q.lexicographic and p.lexicographic
    statuses = _check_rows(bits, dtype, k, p, q, seed=4)
    assert statuses.count(oprofk.STATUS_FILTERED) >= B - 2


def test_lex_rows_constant_values():
    # every draw of every row ties: the tied indices exceed the list kept in
    # LDS, so the draws are visited again
    B, D, k = 8, 4096, 8
    bits = np.full((B, D), 0x3FC0, dtype=np.uint16)    # bf16 1.5
    p = pk.plan_rows(D, k, 1e-3, 1.0, lexicographic=1, S_min=2048, S_max=2048, force_mode=pk.FORCE_FILTER)
    q = oplan.plan_rows(D, k, 1e-3, 1.0, dataclasses.replace(oplan.ROW_OPTS, S_min=2048, S_max=2048,
                                                            force_mode=oplan.FORCE_FILTER, lexicographic=True))
    assert (q.S, q.t, q.M) == (p.S, p.t, p.M)
    statuses = _check_rows(bits, "bf16", k, p, q, seed=11)
    assert all(s == oprofk.STATUS_FILTERED for s in statuses)


def test_lex_rows_config4_256_rows():
    """The C4 batch (bf16 [4096, 131072], k = 32) under the lexicographic
    rule: the whole batch on the GPU, 256 fixed rows checked against the
    oracle (bf16 has few distinct values near the threshold, so ties at tau
    are common), each with its own row stream."""
    b = workloads.relu_normal_bf16((4096, 131072), seed=3)
    B, D, k = b.shape[0], b.shape[1], 32
    p = pk.plan_rows(D, k, 1e-6, 1.0, lexicographic=1)
    q = oplan.plan_rows(D, k, 1e-6, 1.0, dataclasses.replace(oplan.ROW_OPTS, lexicographic=True))
    assert (q.S, q.t, q.M) == (p.S, p.t, p.M) and p.lexicographic
    note(f"lex config4 S={p.S} t={p.t} M={p.M}")
    g = torch().from_numpy(b.view(np.int16)).cuda().view(torch().bfloat16)
    vals, idx, info = pk.topk_rows(g, k, seed=0, p=p)
    torch().cuda.synchronize()
    gv = vals.view(torch().int16).cpu().numpy().view(np.uint16)
    gi = idx.cpu().numpy()
    recs = pk.read_info(info)
    for r in np.arange(0, B, 16):
        ref = oprofk.run(b[r], "bf16", k, q, 0, row=int(r))
        rec = recs[r]
        assert int(rec["status"]) == ref.status, r
        assert int(rec["tau_key"]) == ref.tau_key and int(rec["count"]) == ref.count, r
        assert int(rec["n_valid"]) == ref.n_valid, r
        assert np.array_equal(gi[r], ref.idx), r
        assert np.array_equal(gv[r], ref.vals), r
