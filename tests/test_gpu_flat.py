"""GPU parity of the flat (single-vector) path against the CPU oracle.

Every comparison is bit-exact on values and indices (the method only
compares and copies), and also checks the threshold key, the survivor count
and the status the oracle's stage-by-stage run produces with the same seed.
"""

import numpy as np
import pytest

import paper_2608_12573_amd as pk
import workloads
from oracle import exact, keys as okeys, philox, plan as oplan, profk as oprofk
from gpu_util import (compare, gpu_bf16, gpu_f32, host_bits, note, oracle_plan_of,
                      plan_from_lib, torch)

pytestmark = pytest.mark.gpu


def _f32_case(x, k, seed, eps=1e-6, recall=1.0, offset=0, **kw):
    p = pk.plan(x.size, k, eps, recall, **kw)
    q = oracle_plan_of(p, **kw)
    note(f"flat f32 N={x.size} k={k} seed={seed} off={offset} S={p.S} t={p.t} M={p.M} mode={p.mode}")
    g = gpu_f32(x, offset)
    vals, idx, info = pk.topk(g, k, seed=seed, p=p)
    ref = oprofk.run(okeys.f32_bits(x), "f32", k, q, seed)
    return compare(vals, idx, info, ref, "f32"), ref


def _bf16_case(b, k, seed, eps=1e-6, recall=1.0, offset=0, **kw):
    p = pk.plan(b.size, k, eps, recall, **kw)
    q = oracle_plan_of(p, **kw)
    note(f"flat bf16 N={b.size} k={k} seed={seed} off={offset} S={p.S} t={p.t} M={p.M}")
    g = gpu_bf16(b, offset)
    vals, idx, info = pk.topk(g, k, seed=seed, p=p)
    ref = oprofk.run(b, "bf16", k, q, seed)
    return compare(vals, idx, info, ref, "bf16"), ref


# ----------------------------------------------------------- stage 1 ------
@pytest.mark.parametrize("seed,row,S,N", [(0, 0, 32768, 2**20), (123, 7, 1359, 131072),
                                          (2**63 + 5, 0, 131072, 2**28), (1, 0, 5, 3),
                                          (99, 4095, 4097, 2**32 - 1)])
def test_sample_indices_match_oracle(seed, row, S, N):
    note(f"sample_indices seed={seed} row={row} S={S} N={N}")
    got = pk.debug_sample_indices(seed, row, S, N).cpu().numpy()
    assert np.array_equal(got, philox.sample_indices(seed, row, S, N))


# ----------------------------------------------------------- stage 3 ------
@pytest.mark.parametrize("offset", [0, 1, 2, 3])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_filter_survivor_set(dtype, offset):
    N = 3 * 2**20 + 5
    if dtype == "f32":
        x = workloads.normal_f32(N, seed=11)
        bits = okeys.f32_bits(x)
        g = gpu_f32(x, offset)
    else:
        bits = workloads.relu_normal_bf16(N, seed=11)
        g = gpu_bf16(bits, offset)
    key = okeys.keys_of(bits, dtype)
    tau = int(np.sort(key)[-5000])                         # about 5000 survivors
    p = pk.plan(N, 64, 1e-6, 1.0, S_min=4096, S_max=4096, force_mode=pk.FORCE_FILTER)
    p.M = 20000
    surv = oprofk.survivors(key, tau)
    for rep in range(3):
        note(f"debug_filter {dtype} N={N} off={offset} rep={rep}")
        bk, bi, cnt = pk.debug_filter(g, tau, p)
        n = int(cnt.cpu().numpy()[0])
        assert n == surv.size
        gi = bi.cpu().numpy().view(np.uint32)[:n].astype(np.int64)
        gk = bk.cpu().numpy().view(np.uint32)[:n].astype(np.int64)
        order = np.argsort(gi)
        assert np.array_equal(gi[order], surv)
        assert np.array_equal(gk[order], key[surv])


def test_filter_counts_past_capacity():
    N = 2**20 + 3
    x = workloads.uniform_f32(N, seed=12)
    key = okeys.keys_of(okeys.f32_bits(x), "f32")
    p = pk.plan(N, 64, 1e-6, 1.0, S_min=4096, S_max=4096, force_mode=pk.FORCE_FILTER)
    p.M = 100
    tau = int(np.sort(key)[-100000])
    note("debug_filter past capacity")
    bk, bi, cnt = pk.debug_filter(gpu_f32(x), tau, p)
    assert int(cnt.cpu().numpy()[0]) == 100000
    gi = bi.cpu().numpy().view(np.uint32)[:100].astype(np.int64)
    assert np.all(key[gi] >= tau) and np.unique(gi).size == 100


# ------------------------------------------------------------ end to end --
@pytest.mark.parametrize("seed", range(10))
def test_config1_uniform_2p20_k64(seed):
    x = workloads.uniform_f32(2**20, seed=0)
    rec, ref = _f32_case(x, 64, seed)
    assert ref.status == oprofk.STATUS_FILTERED


SMALL = dict(S_min=2048, S_max=2048, force_mode=pk.FORCE_FILTER)


@pytest.mark.parametrize("N,k", [(5000, 1), (5000, 7), (65536 + 17, 64), (65536 + 17, 1000),
                                 (300_001, 4096), (1 << 20, 333), (4099, 4096)])
@pytest.mark.parametrize("dist", ["normal", "uniform", "ints"])
def test_small_sizes_forced_filter(N, k, dist):
    g = np.random.default_rng(N + k)
    x = {"normal": lambda: g.standard_normal(N).astype(np.float32),
         "uniform": lambda: g.random(N, dtype=np.float32),
         "ints": lambda: g.integers(0, 300, N).astype(np.float32)}[dist]()
    for seed in range(3):
        _f32_case(x, k, seed, eps=1e-3, **SMALL)


@pytest.mark.parametrize("offset", [1, 2, 3])
def test_unaligned_base(offset):
    x = workloads.normal_f32(2**20 + 9, seed=3)
    _f32_case(x, 100, 5, offset=offset)


def test_special_values_and_ties():
    x = workloads.special_f32(200_000, seed=6)
    for k in (1, 10, 500, 4096):
        _f32_case(x, k, 1, eps=1e-3, **SMALL)


# Plans with t > 32: sample blocks keep lists of their largest draws and
# one block selects tau from the union of those lists (k_select_tau).  Two
# regimes, told apart by mu = 1024 t / S, the mean number of a 1024-draw
# block's draws in the sample's top t: at k = 4096 (mu about 5) blocks of
# 1024 draws keep capped lists of 32 and the select checks them against
# their cut keys, falling back to all sample keys on ties; at k = 8192 (mu
# about 10) blocks of 4096 draws keep their whole top t.  A constant input
# makes every key equal (the select's shared-prefix trim takes all bits),
# small integers leave thousands of ties in the union, S = 40002 leaves a
# partial last sample block (66 draws with capped lists: not a multiple of
# a thread's four, so the last keys are stored one by one).
@pytest.mark.parametrize("case", ["normal", "constant", "ints", "S40002", "bf16"])
@pytest.mark.parametrize("k", [4096, 8192])
@pytest.mark.parametrize("seed", [0, 3])
def test_large_t_threshold(case, k, seed):
    N = 2**20
    rng = np.random.default_rng(31)

    def regime(p):
        mu = 1024 * p.t / p.S
        assert p.t > 32 and (mu < 6 if k == 4096 else mu > 7), (p.S, p.t)

    if case == "bf16":
        kb = 2048 if k == 4096 else 8192
        b = workloads.relu_normal_bf16(N, seed=31)
        p = pk.plan(N, kb, 1e-3, 1.0)
        regime(p)
        q = oracle_plan_of(p)
        note(f"large t bf16 N={N} k={kb} seed={seed} S={p.S} t={p.t}")
        vals, idx, info = pk.topk(gpu_bf16(b), kb, seed=seed, p=p)
        compare(vals, idx, info, oprofk.run(b, "bf16", kb, q, seed), "bf16")
        return
    x = {"normal": lambda: rng.standard_normal(N).astype(np.float32),
         "constant": lambda: np.full(N, 1.5, dtype=np.float32),
         "ints": lambda: rng.integers(0, 300, N).astype(np.float32),
         "S40002": lambda: rng.standard_normal(N).astype(np.float32)}[case]()
    kw = dict(S_min=40002, S_max=40002) if case == "S40002" else {}
    regime(pk.plan(N, k, 1e-3, 1.0, **kw))
    rec, ref = _f32_case(x, k, seed, eps=1e-3, **kw)


@pytest.mark.parametrize("k,plateau,value", [(1024, 1000, 3.2), (4096, 2800, 3.0)])
def test_tie_plateau_at_rank_k(k, plateau, value):
    # a plateau of equal values where rank k falls: one log-scale bucket at
    # or above rank k holds the whole plateau, far more than 128 candidates;
    # the one-workgroup refinement ranks it by comparison (ties by index)
    x = workloads.normal_f32(2**20, seed=12)
    rng = np.random.default_rng(12)
    x[rng.choice(x.size, plateau, replace=False)] = np.float32(value)
    rec, ref = _f32_case(x, k, 0)
    assert ref.status == oprofk.STATUS_FILTERED


@pytest.mark.parametrize("N,k", [(1, 1), (3, 2), (64, 64), (1000, 10), (1000, 1000), (30_000, 4096)])
def test_direct_mode(N, k):
    x = workloads.special_f32(N, seed=N)
    rec, ref = _f32_case(x, k, 0)
    assert ref.status == oprofk.STATUS_DIRECT


@pytest.mark.parametrize("offset", [0, 1, 3])
def test_bf16_flat(offset):
    b = workloads.relu_normal_bf16(2**20 + 11, seed=3)
    for k in (32, 100, 4096):
        _bf16_case(b, k, 2, offset=offset)


def test_relaxed_recall_flat():
    x = workloads.normal_f32(2**20, seed=8)
    for seed in range(5):
        rec, ref = _f32_case(x, 2000, seed, recall=0.9)


@pytest.mark.parametrize("survivors", [1900, 1801])
def test_relaxed_partial_output_small_k(survivors):
    # k_req <= count < k at k <= 4096: every candidate is refined (rank k
    # lies past them), shared out among several refining workgroups, and
    # workgroup 0 writes the padding after the count
    x = workloads.normal_f32(2**20, seed=26)
    bits = okeys.f32_bits(x)
    key = np.sort(okeys.key_u32(bits).astype(np.int64))
    k = 2000
    p = pk.plan(x.size, k, 1e-3, 0.9, S_min=8192, S_max=8192, force_mode=pk.FORCE_FILTER)
    q = plan_from_lib(p)
    tau = int(key[-survivors])
    note(f"flat relaxed partial k={k} survivors={survivors} k_req={p.k_req}")
    vals, idx, info = pk.topk_tau(gpu_f32(x), k, tau, p)
    ref = oprofk.run(bits, "f32", k, q, 0, tau_override=tau)
    assert ref.status == oprofk.STATUS_FILTERED and ref.n_valid == survivors
    compare(vals, idx, info, ref, "f32")


# ------------------------------------------------------- forced failures --
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_forced_underflow_and_overflow(dtype):
    N = 500_000
    if dtype == "f32":
        x = workloads.uniform_f32(N, seed=9)
        x[[5, 77, 1234]] = 2.0
        bits = okeys.f32_bits(x)
        g = gpu_f32(x)
    else:
        bits = workloads.relu_normal_bf16(N, seed=9)
        g = gpu_bf16(bits)
    key = okeys.keys_of(bits, dtype)
    k = 64
    p = pk.plan(N, k, 1e-6, 1.0, S_min=4096, S_max=4096, force_mode=pk.FORCE_FILTER)
    q = plan_from_lib(p)
    for tau, want in ((int(key.max()), oprofk.STATUS_UNDERFLOW), (int(key.min()), oprofk.STATUS_OVERFLOW)):
        note(f"topk_tau {dtype} tau={tau:#x}")
        vals, idx, info = pk.topk_tau(g, k, tau, p)
        ref = oprofk.run(bits, dtype, k, q, 0, tau_override=tau)
        assert ref.status == want
        compare(vals, idx, info, ref, dtype)


def test_plan_override_small_buffer_overflows():
    x = workloads.normal_f32(2**20, seed=10)
    p = pk.plan(2**20, 64)
    p.M = 64
    q = plan_from_lib(p)
    note("plan override M=k")
    vals, idx, info = pk.topk(gpu_f32(x), 64, seed=0, p=p)
    ref = oprofk.run(okeys.f32_bits(x), "f32", 64, q, 0)
    assert ref.status == oprofk.STATUS_OVERFLOW
    compare(vals, idx, info, ref, "f32")


def test_repeat_is_deterministic():
    x = workloads.normal_f32(2**22, seed=13)
    g = gpu_f32(x)
    p = pk.plan(x.size, 256)
    note("determinism x20")
    first = None
    for _ in range(20):
        vals, idx, info = pk.topk(g, 256, seed=4, p=p)
        cur = (host_bits(vals).tobytes(), idx.cpu().numpy().tobytes(), info.cpu().numpy().tobytes())
        if first is None:
            first = cur
        assert cur == first


def test_simple_entry_point():
    x = workloads.normal_f32(2**20, seed=14)
    note("topk_simple")
    vals, idx = pk.topk_simple(gpu_f32(x), 50, seed=3)
    v, i = exact.topk(okeys.f32_bits(x), "f32", 50)
    assert np.array_equal(idx.cpu().numpy(), i)
    assert np.array_equal(host_bits(vals), v)
    pk.lib().profk_release()


# ------------------------------------------------------ full-size configs --
@pytest.fixture(scope="module")
def c2_input():
    return workloads.normal_f32(2**28, seed=1)


@pytest.mark.parametrize("k", [16, 256, 1024, 4096])
def test_config2_normal_2p28(c2_input, k):
    rec, ref = _f32_case(c2_input, k, 0)
    assert ref.status == oprofk.STATUS_FILTERED


C3 = {"pareto": lambda n: workloads.pareto_f32(n, seed=2),
      "zeros90": lambda n: workloads.zeros90_f32(n, seed=2),
      "ramp": lambda n: workloads.ramp_f32(n),
      "plateau": lambda n: workloads.plateau_f32(n, seed=2, width=10_000),
      "plateau_wide": lambda n: workloads.plateau_f32(n, seed=2, width=200_000)}


@pytest.mark.parametrize("name", list(C3))
def test_config3_adversarial_2p26(name):
    x = C3[name](2**26)
    rec, ref = _f32_case(x, 512, 0)
    if name == "plateau_wide":
        assert ref.status == oprofk.STATUS_OVERFLOW


# ------------------------------------------------------- sorted inputs ----
# The filter deals tiles of the input to its workgroups in turn, so the
# survivors of a sorted input sit in the first or last tiles: a few
# workgroups hold them all, at either end of the grid, next to the ragged
# head and tail outside the 16-byte vectors.
@pytest.mark.parametrize("descending", [False, True])
@pytest.mark.parametrize("k", [100, 4096])
@pytest.mark.parametrize("offset", [0, 3])
def test_sorted_f32_unaligned(descending, k, offset):
    n = 3 * (1 << 20) + 7
    x = workloads.ramp_f32(n)
    if descending:
        x = x[::-1].copy()
    rec, ref = _f32_case(x, k, 5, offset=offset)
    assert ref.status == oprofk.STATUS_FILTERED


@pytest.mark.parametrize("descending", [False, True])
def test_sorted_bf16_unaligned(descending):
    # a ramp of fp32 in (0, 1] rounded to bf16: runs of equal values, the
    # top one (1.0) about 4096 long, so the k-th key is cut in index order
    n = (1 << 22) + 5
    b = workloads.f32_to_bf16_bits(((np.arange(n, dtype=np.float64) + 1) / n).astype(np.float32))
    if descending:
        b = b[::-1].copy()
    _bf16_case(b, 1000, 6, offset=1)
