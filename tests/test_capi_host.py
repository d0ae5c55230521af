"""Host-side checks of libprofk.so (no GPU needed): every symbol the header
declares is exported, the C++ planner equals the oracle planner, and bad
arguments are rejected with the documented codes."""

import itertools
import math

import pytest

import paper_2608_12573_amd as pk
from oracle import plan as oplan


def test_library_exports_every_header_symbol():
    L = pk.lib()
    names = pk.header_functions()
    assert len(names) >= 15
    for name in names:
        assert hasattr(L, name), name


def _oracle_opts(o):
    return oplan.PlanOpts(S_min=o.S_min, S_max=o.S_max, cost_ratio=o.cost_ratio,
                          eps_split=o.eps_split, paper_literal=bool(o.paper_literal),
                          force_mode=o.force_mode, lexicographic=bool(o.lexicographic))


def _same(p, q):
    assert (p.N, p.k, p.k_req, p.S, p.t, p.M, p.mode) == (q.N, q.k, q.k_req, q.S, q.t, q.M, q.mode)
    assert bool(p.lexicographic) == q.lexicographic
    assert p.p_underflow == pytest.approx(q.p_underflow, rel=1e-9, abs=1e-300)
    assert p.p_overflow == pytest.approx(q.p_overflow, rel=1e-9, abs=1e-300)


GRID_N = [1000, 4096, 65537, 2**20, 3 * 10**6, 2**24 + 3, 2**26, 2**28, 2**30, 2**32 - 1]
GRID_K = [1, 2, 16, 64, 512, 1024, 4096, 65536, 262144]
GRID_E = [1e-1, 1e-3, 1e-6, 1e-9]
GRID_R = [1.0, 0.95, 0.5]


@pytest.mark.parametrize("N", GRID_N)
def test_planner_equals_oracle_grid(N):
    for k, eps, rho in itertools.product(GRID_K, GRID_E, GRID_R):
        if k > N:
            continue
        p = pk.plan(N, k, eps, rho)
        q = oplan.plan(N, k, eps, rho)
        _same(p, q)


@pytest.mark.parametrize("D", [4096, 131072, 65536, 12288])
def test_row_planner_equals_oracle(D):
    for k in (1, 8, 32, 64, 256):
        for eps in (1e-6, 1e-3):
            p = pk.plan_rows(D, k, eps)
            q = oplan.plan_rows(D, k, eps)
            _same(p, q)


@pytest.mark.parametrize("B,d_dict,k_row", [(4096, 12288, 32), (4096, 65536, 64), (256, 2048, 8), (64, 512, 4)])
def test_sae_planner_equals_oracle(B, d_dict, k_row):
    for eps, recall in ((1e-6, 1.0), (1e-3, 0.95)):
        p = pk.plan_sae(B, d_dict, k_row, eps, recall)
        q = oplan.plan(B * d_dict, B * k_row, eps, recall, oplan.SAE_OPTS)
        _same(p, q)


def test_paper_literal_and_options_equal_oracle():
    cases = [dict(paper_literal=1), dict(S_min=64, S_max=64, force_mode=pk.FORCE_FILTER), dict(lexicographic=1),
             dict(cost_ratio=0.1), dict(eps_split=0.3), dict(S_min=131072, S_max=131072)]
    for kw, (N, k) in itertools.product(cases, [(2**20, 64), (2**28, 1024), (2**29, 64),
                                                (10**6, 10), (2**28, 262144)]):
        o = pk.opts(True, **kw)
        p = pk.plan(N, k, 1e-6, 1.0, **kw)
        q = oplan.plan(N, k, 1e-6, 1.0, _oracle_opts(o))
        _same(p, q)


def test_plan_rejects_bad_arguments():
    bad = [(0, 1, 1e-6, 1.0), (10, 0, 1e-6, 1.0), (10, 11, 1e-6, 1.0), (10, 5, 0.0, 1.0),
           (10, 5, 1.0, 1.0), (10, 5, 1e-3, 0.0), (10, 5, 1e-3, 1.5), (2**32, 5, 1e-3, 1.0)]
    for N, k, e, r in bad:
        with pytest.raises(pk.ProfkError, match="invalid argument"):
            pk.plan(N, k, e, r)
    with pytest.raises(pk.ProfkError):
        pk.plan(100, 5, 1e-3, 1.0, S_min=0)


def test_workspace_is_small_and_validates():
    p = pk.plan(2**28, 1024)
    ws = pk.workspace_size(p, pk.F32)
    assert 0 < ws < 64 << 20          # O(S + M + k), far below the 1 GiB input
    assert pk.workspace_size(p, 7) == 0
    assert pk.workspace_size(p, pk.F32, 0) == 0


def test_status_strings():
    L = pk.lib()
    for code in (pk.OK, pk.EINVAL, pk.EDTYPE, pk.EWORKSPACE, pk.ENULL, pk.EHIP, 12345):
        assert L.profk_status_string(code)


def test_null_and_dtype_errors_without_gpu():
    L = pk.lib()
    p = pk.plan(2**20, 64)
    import ctypes
    rc = L.profk_topk(ctypes.byref(p), pk.F32, None, 2**20, 64, 0, None, None, None, 0, None, None)
    assert rc == pk.ENULL
    rc = L.profk_topk(ctypes.byref(p), 9, ctypes.c_void_p(16), 2**20, 64, 0, ctypes.c_void_p(16),
                      ctypes.c_void_p(16), ctypes.c_void_p(16), 1 << 30, None, None)
    assert rc == pk.EDTYPE
    rc = L.profk_topk(ctypes.byref(p), pk.F32, ctypes.c_void_p(16), 2**20, 65, 0, ctypes.c_void_p(16),
                      ctypes.c_void_p(16), ctypes.c_void_p(16), 1 << 30, None, None)
    assert rc == pk.EINVAL
    rc = L.profk_topk(ctypes.byref(p), pk.F32, ctypes.c_void_p(16), 2**20, 64, 0, ctypes.c_void_p(16),
                      ctypes.c_void_p(16), ctypes.c_void_p(16), 16, None, None)
    assert rc == pk.EWORKSPACE
    rc = L.profk_topk(ctypes.byref(p), pk.F32, ctypes.c_void_p(18), 2**20, 64, 0, ctypes.c_void_p(16),
                      ctypes.c_void_p(16), ctypes.c_void_p(16), 1 << 30, None, None)
    assert rc == pk.EINVAL


def test_oracle_and_product_share_no_code():
    import os
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    for d, needle in (("oracle", "paper_2608_12573_amd"), ("paper_2608_12573_amd", "oracle")):
        for dirpath, _, files in os.walk(os.path.join(root, d)):
            if "_build" in dirpath:
                continue
            for fn in files:
                if fn.endswith((".py", ".hip", ".cpp", ".h")):
                    with open(os.path.join(dirpath, fn)) as f:
                        text = f.read()
                    assert f"import {needle}" not in text and f"from {needle}" not in text, fn
                    assert f"{needle}/" not in text, fn


def test_binding_shares_torchs_hip_runtime():
    # A fresh process that loads the library through the binding must end up
    # with a single HIP runtime (torch's), whatever it touches first.
    import subprocess
    import sys
    code = (
        "import os, sys\n"
        f"sys.path.insert(0, {repr(__import__('os').path.dirname(__import__('os').path.dirname(__import__('os').path.abspath(__file__))))})\n"
        "import paper_2608_12573_amd as pk\n"
        "pk.plan(1 << 20, 64)\n"
        "import torch\n"
        "maps = open('/proc/self/maps').read()\n"
        "libs = sorted(set(l.split()[-1] for l in maps.splitlines() if 'libamdhip64' in l))\n"
        "print(len(libs)); print(libs)\n"
    )
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stderr
    assert out.stdout.splitlines()[0] == "1", out.stdout


def test_rows_workspace_and_refusals_outside_the_row_kernel():
    """Row plans the one-workgroup kernel takes need no workspace; larger
    ones need one row's vector workspace, and the call refuses a missing
    or short one before anything is enqueued (host-only checks)."""
    import ctypes
    fits = pk.plan_rows(131072, 32)
    wide = pk.plan_rows(2**22, 32)
    big_k = pk.plan_rows(65536, 2048)
    assert pk.workspace_size(fits, pk.BF16, 4096) == 256
    for p in (wide, big_k):
        need = pk.workspace_size(p, pk.F32, 8)
        assert need == pk.workspace_size(p, pk.F32, 1) > 256
    L = pk.lib()
    dummy = ctypes.c_void_p(256)   # never dereferenced: the calls fail their host checks
    rc = L.profk_topk_rows(ctypes.byref(wide), pk.F32, dummy, 8, 2**22, 2**22, 32, 0, dummy, dummy,
                           None, 0, None, None)
    assert rc == pk.ENULL
    rc = L.profk_topk_rows(ctypes.byref(wide), pk.F32, dummy, 8, 2**22, 2**22, 32, 0, dummy, dummy,
                           dummy, pk.workspace_size(wide, pk.F32, 8) - 1, None, None)
    assert rc == pk.EWORKSPACE
    # a plan whose buffer words would wrap the row kernel's 32-bit LDS sums
    huge = pk.plan_rows(2**32 - 1, 16, S_min=1, S_max=1, force_mode=pk.FORCE_FILTER)
    assert huge.M > 2**30
    assert pk.workspace_size(huge, pk.F32, 2) > 256


def test_read_probe_refuses_bad_arguments():
    """Host-side checks of profk_debug_read_probe; the dummy pointers are
    never dereferenced because every call fails before a launch."""
    import ctypes
    L = pk.lib()
    ptr, out = ctypes.c_void_p(4096), ctypes.c_void_p(8192)
    grid = ctypes.c_uint32(0)
    assert L.profk_debug_read_probe(ptr, 100, 2, 4, out, ctypes.byref(grid), None) == pk.EINVAL      # not 16-byte multiple
    assert L.profk_debug_read_probe(ctypes.c_void_p(4100), 4096, 2, 4, out, ctypes.byref(grid), None) == pk.EINVAL
    assert L.profk_debug_read_probe(ptr, 4096, 0, 4, out, ctypes.byref(grid), None) == pk.EINVAL
    assert L.profk_debug_read_probe(ptr, 4096, 2, 5, out, ctypes.byref(grid), None) == pk.EINVAL
    assert L.profk_debug_read_probe(ptr, 16 * (2**32 - 2**22), 2, 4, out, ctypes.byref(grid), None) == pk.EINVAL
    assert L.profk_debug_read_probe(None, 4096, 2, 4, out, ctypes.byref(grid), None) == pk.ENULL
