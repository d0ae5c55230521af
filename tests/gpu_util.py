"""Helpers shared by the GPU parity tests: moving seeded inputs to the GPU,
reading results back as bit patterns, and running the oracle under the same
plan the library chose (after checking the two planners agree)."""

import sys

import numpy as np

import paper_2608_12573_amd as pk
from oracle import keys as okeys
from oracle import plan as oplan
from oracle import profk as oprofk


def torch():
    import torch as t
    return t


def note(msg):
    """Name the case before a GPU step, flushed, so a failed run shows it."""
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def gpu_f32(x, offset=0):
    """fp32 CUDA tensor view of x, optionally starting `offset` elements into
    a larger allocation (to test unaligned bases)."""
    t = torch()
    x = np.ascontiguousarray(x, dtype=np.float32)
    if offset == 0:
        return t.from_numpy(x).cuda()
    big = t.empty(x.size + offset, dtype=t.float32, device="cuda")
    big[offset:] = t.from_numpy(x).cuda()
    return big[offset:]


def gpu_bf16(bits_u16, offset=0):
    t = torch()
    b = np.ascontiguousarray(bits_u16, dtype=np.uint16).view(np.int16)
    g = t.from_numpy(b).cuda().view(t.bfloat16)
    if offset == 0:
        return g
    big = t.empty(g.numel() + offset, dtype=t.bfloat16, device="cuda")
    big[offset:] = g
    return big[offset:]


def host_bits(tensor):
    t = torch()
    if tensor.dtype == t.float32:
        return tensor.contiguous().view(t.int32).cpu().numpy().view(np.uint32)
    if tensor.dtype == t.bfloat16:
        return tensor.contiguous().view(t.int16).cpu().numpy().view(np.uint16)
    raise TypeError(tensor.dtype)


def oracle_plan_of(p, opts=None, rows=False, **kw):
    """The oracle's own plan for the same request, asserted equal to the
    library's plan p (the planners are independent implementations)."""
    o = opts if opts is not None else oplan.PlanOpts(**kw) if kw else (oplan.ROW_OPTS if rows else oplan.PlanOpts())
    q = oplan.plan(p.N, p.k, p.eps, p.recall, o)
    assert (q.S, q.t, q.M, q.k_req, q.mode) == (p.S, p.t, p.M, p.k_req, p.mode), (q, p.as_dict())
    assert q.lexicographic == bool(p.lexicographic)
    return q


def plan_from_lib(p):
    """oracle Plan carrying exactly the library plan's numbers (used when a
    test edits a plan on purpose)."""
    return oplan.Plan(N=p.N, k=p.k, eps=p.eps, recall=p.recall, k_req=p.k_req, S=p.S, t=p.t, M=p.M,
                      mode=p.mode, p_underflow=p.p_underflow, p_overflow=p.p_overflow,
                      lexicographic=bool(p.lexicographic))


def compare(vals, idx, info, ref, dtype):
    """Bit-exact comparison of a GPU result with an oracle Result."""
    gv = host_bits(vals)
    gi = idx.cpu().numpy()
    rec = pk.read_info(info)[0]
    assert int(rec["status"]) == ref.status, (int(rec["status"]), ref.status)
    assert int(rec["n_valid"]) == ref.n_valid
    if ref.status != oprofk.STATUS_DIRECT:
        assert int(rec["tau_key"]) == ref.tau_key, (hex(int(rec["tau_key"])), hex(ref.tau_key))
        assert int(rec["count"]) == ref.count, (int(rec["count"]), ref.count)
    bad = np.flatnonzero(gi != ref.idx)
    assert bad.size == 0, f"{bad.size} index mismatches, first at {bad[:5]}: gpu {gi[bad[:5]]} ref {ref.idx[bad[:5]]}"
    assert np.array_equal(gv, ref.vals)
    return rec


def keys_of(bits, dtype):
    return okeys.keys_of(bits, dtype)


def check_rows(bits2d, dtype, k, p, q, seed, offset=0, stride=None):
    """Per-row parity: the library's profk_topk_rows against the oracle run
    row by row (each row its own Philox stream), bit-exact, with every row's
    threshold, count, status and n_valid.  Returns the oracle statuses."""
    t = torch()
    B, D = bits2d.shape
    stride = D if stride is None else stride
    padded = np.zeros((B, stride), dtype=bits2d.dtype)
    padded[:, :D] = bits2d
    flat = padded.reshape(-1)
    g = gpu_f32(flat.view(np.float32), offset) if dtype == "f32" else gpu_bf16(flat, offset)
    x = g.view(B, stride)[:, :D]
    note(f"rows {dtype} B={B} D={D} stride={stride} off={offset} k={k} S={p.S} t={p.t} M={p.M}")
    vals, idx, info = pk.topk_rows(x, k, seed=seed, p=p)
    t.cuda.synchronize()
    gv = host_bits(vals).reshape(B, k)
    gi = idx.cpu().numpy().reshape(B, k)
    recs = pk.read_info(info)
    statuses = []
    for r in range(B):
        ref = oprofk.run(bits2d[r], dtype, k, q, seed, row=r)
        statuses.append(ref.status)
        rec = recs[r]
        assert int(rec["status"]) == ref.status, (r, int(rec["status"]), ref.status)
        if ref.status != oprofk.STATUS_DIRECT:
            assert int(rec["tau_key"]) == ref.tau_key, r
            assert int(rec["count"]) == ref.count, r
        assert int(rec["n_valid"]) == ref.n_valid, r
        assert np.array_equal(gi[r], ref.idx), (r, gi[r][:8], ref.idx[:8])
        assert np.array_equal(gv[r], ref.vals), r
    return statuses
