"""profk_topk_noalloc against profk_topk, called through the C ABI.

The no-allocation entry point runs the same kernels on the library's fixed
per-GPU scratch array instead of a caller's workspace, so its outputs and
reports must equal profk_topk's bit for bit.  Two calls run back to back,
the second on a smaller input, so the second reads a scratch array the
first left full of its own state; an all-equal input drives the exact
fallback, whose tickets live in the same array.
"""

import ctypes

import numpy as np
import pytest

import paper_2608_12573_amd as pk
import workloads
from oracle import keys as okeys, profk as oprofk
from gpu_util import compare, gpu_bf16, gpu_f32, host_bits, note, oracle_plan_of, torch

pytestmark = pytest.mark.gpu


def _noalloc_raw(x, k, p, seed):
    """One profk_topk_noalloc call straight through ctypes."""
    t = torch()
    vals = t.empty(k, dtype=x.dtype, device=x.device)
    idx = t.empty(k, dtype=t.int64, device=x.device)
    info = t.empty(pk.INFO_BYTES, dtype=t.uint8, device=x.device)
    dt = pk.F32 if x.dtype == t.float32 else pk.BF16
    stream = ctypes.c_void_p(t.cuda.current_stream().cuda_stream)
    rc = pk.lib().profk_topk_noalloc(ctypes.byref(p), dt, ctypes.c_void_p(x.data_ptr()), x.numel(), k, seed,
                                     ctypes.c_void_p(vals.data_ptr()), ctypes.c_void_p(idx.data_ptr()), stream,
                                     ctypes.c_void_p(info.data_ptr()))
    assert rc == pk.OK, pk.lib().profk_status_string(rc)
    return vals, idx, info


def _same(a, b):
    """Equal outputs and reports of two calls (values as bit patterns)."""
    assert np.array_equal(host_bits(a[0]), host_bits(b[0]))
    assert np.array_equal(a[1].cpu().numpy(), b[1].cpu().numpy())
    ra, rb = pk.read_info(a[2])[0], pk.read_info(b[2])[0]
    for f in ("count", "tau_key", "status", "n_valid"):
        assert int(ra[f]) == int(rb[f]), (f, int(ra[f]), int(rb[f]))


def _pair(x, k, seed, ref_bits=None, dtype="f32"):
    p = pk.plan(x.numel(), k)
    assert pk.workspace_size(p, pk.F32 if dtype == "f32" else pk.BF16) <= pk.NOALLOC_SCRATCH_BYTES
    note(f"noalloc {dtype} N={x.numel()} k={k} seed={seed}")
    got = _noalloc_raw(x, k, p, seed)
    want = pk.topk(x, k, seed=seed, p=p)
    torch().cuda.synchronize()
    _same(got, want)
    if ref_bits is not None:
        ref = oprofk.run(ref_bits, dtype, k, oracle_plan_of(p), seed)
        compare(got[0], got[1], got[2], ref, dtype)
    return pk.read_info(got[2])[0]


def test_noalloc_two_calls_larger_then_smaller():
    x1 = workloads.normal_f32(2**24 + 3, seed=21)
    x2 = workloads.uniform_f32(2**20 + 7, seed=22)
    g1, g2 = gpu_f32(x1, offset=1), gpu_f32(x2)
    r1 = _pair(g1, 4096, 3, okeys.f32_bits(x1))
    r2 = _pair(g2, 64, 4, okeys.f32_bits(x2))
    assert int(r1["status"]) == oprofk.STATUS_FILTERED and int(r2["status"]) == oprofk.STATUS_FILTERED


def test_noalloc_bf16_then_fallback():
    b = workloads.relu_normal_bf16(3 * 2**20 + 1, seed=23)
    _pair(gpu_bf16(b), 256, 5, b, "bf16")
    # every value equal: the filter overflows and the exact fallback runs,
    # with tickets and merge buffers in the scratch the previous call used
    x = np.full(2**21 + 5, 1.5, dtype=np.float32)
    r = _pair(gpu_f32(x), 100, 6, okeys.f32_bits(x))
    assert int(r["status"]) == oprofk.STATUS_OVERFLOW


def test_noalloc_rejects_plans_beyond_the_scratch():
    """A plan whose workspace exceeds the fixed array is refused before
    anything is enqueued."""
    t = torch()
    x = t.empty(1, dtype=t.float32, device="cuda")
    p = pk.plan(2**28, 262144)
    assert pk.workspace_size(p, pk.F32) > pk.NOALLOC_SCRATCH_BYTES
    out = t.empty(1, dtype=t.float32, device="cuda")
    rc = pk.lib().profk_topk_noalloc(ctypes.byref(p), pk.F32, ctypes.c_void_p(x.data_ptr()), 2**28, 262144, 0,
                                     ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(out.data_ptr()), None, None)
    assert rc == pk.EWORKSPACE
