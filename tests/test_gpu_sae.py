"""GPU parity of the BatchTopK SAE layer (encoder GEMM with the fused
filter, selection, sparse decode) against the fp64 oracle (oracle.sae).

The GPU sums bf16 products in fp32 on the matrix cores, one rounding per
16-product step (and its accumulator) plus one for the bias, so a latent
may differ from the exact value by at most
    tol = (2 * d_model / 16 + 2) * 2^-24 * (sum_m |x w| + |b|).
Selections are compared modulo that: every selected latent equals the exact
value within tol, and the selected and exact sets differ only by latents
within 2 tol_max of the K-th exact value (near-ties under rounding)."""

import numpy as np
import pytest

import paper_2608_12573_amd as pk
import workloads
from oracle import sae as osae
from gpu_util import note, torch

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


def _dev(m):
    t = torch()
    bf = lambda a: t.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(t.bfloat16)
    return dict(x=bf(m["x"]), w_enc=bf(m["w_enc"]), b_enc=t.from_numpy(m["b_enc"]).cuda(),
                w_dec=bf(m["w_dec"]), b_dec=t.from_numpy(m["b_dec"]).cuda())


def _tol(m):
    d_model = m["x"].shape[1]
    return (2 * d_model / 16 + 2) * U * osae.encode_scale(m["x"], m["w_enc"], m["b_enc"])


def _check_selection(vals, idx, z, tol, K):
    """vals/idx: the GPU's selection; z, tol: exact latents and bounds."""
    zf, tf = z.reshape(-1), tol.reshape(-1)
    n_valid = int((idx >= 0).sum())
    assert n_valid == K
    assert np.unique(idx).size == K
    assert np.all(np.abs(vals - zf[idx]) <= tf[idx]), "a selected latent differs from its exact value"
    # sorted under the total order
    assert np.all(vals[:-1] >= vals[1:])
    same = vals[:-1] == vals[1:]
    assert np.all(idx[:-1][same] < idx[1:][same])
    ev, ei = osae.batchtopk(z, K)
    kth, tmax = ev[-1], tf.max()
    gpu_only = np.setdiff1d(idx, ei)
    exact_only = np.setdiff1d(ei, idx)
    assert gpu_only.size == exact_only.size
    assert np.all(zf[gpu_only] >= kth - 2 * tmax)
    assert np.all(zf[exact_only] <= kth + 2 * tmax)
    return gpu_only.size


@pytest.mark.parametrize("B,d_model,d_dict", [(200, 128, 300), (256, 512, 1024), (1, 64, 129), (300, 192, 700)])
def test_sae_dense_latents(B, d_model, d_dict):
    m = workloads.sae_model(B=B, d_model=d_model, d_dict=d_dict, seed=B + d_dict)
    note(f"sae dense B={B} d_model={d_model} d_dict={d_dict}")
    g = _dev(m)
    z_gpu = pk.sae_encode_dense(g["x"], g["w_enc"], g["b_enc"]).cpu().numpy().astype(np.float64)
    z = osae.encode(m["x"], m["w_enc"], m["b_enc"])
    assert np.all(np.abs(z_gpu - z) <= _tol(m))
    assert np.all(z_gpu >= 0) and not np.any(np.signbit(z_gpu))   # +0.0 for inactive latents


def test_sae_sampled_latents_are_the_gemm_values():
    # internal consistency: stage 1 computes each draw's latent with the GEMM's
    # own MFMA sequence, so its key equals the dense latent's key bit for bit
    t = torch()
    B, d_model, d_dict = 256, 512, 2048
    m = workloads.sae_model(B=B, d_model=d_model, d_dict=d_dict, seed=7)
    g = _dev(m)
    p = pk.plan(B * d_dict, B * 16, 1e-6, 1.0, S_min=4096, S_max=4096, force_mode=pk.FORCE_FILTER)
    note(f"sae sample S={p.S}")
    keys = pk.debug_sae_sample(g["x"], g["w_enc"], g["b_enc"], p, seed=3).cpu().numpy()
    idx = pk.debug_sample_indices(3, 0, p.S, B * d_dict).cpu().numpy()
    dense = pk.sae_encode_dense(g["x"], g["w_enc"], g["b_enc"]).reshape(-1)
    bits = dense.view(t.int32).cpu().numpy().astype(np.int64) & 0xFFFFFFFF
    assert np.array_equal(keys, bits[idx] ^ 0x80000000)     # latents are >= +0: key = bits with the sign set


@pytest.mark.parametrize("B,d_model,d_dict,k_row", [(256, 512, 2048, 32), (300, 128, 1000, 8), (128, 256, 4096, 4),
                                                   (200, 192, 700, 8), (64, 64, 513, 4)])
def test_sae_encode_topk(B, d_model, d_dict, k_row):
    m = workloads.sae_model(B=B, d_model=d_model, d_dict=d_dict, seed=11)
    g = _dev(m)
    K = B * k_row
    p = pk.plan(B * d_dict, K)
    note(f"sae topk B={B} d_model={d_model} d_dict={d_dict} K={K} S={p.S} t={p.t} M={p.M} mode={p.mode}")
    vals, idx, info = pk.sae_encode_topk(g["x"], g["w_enc"], g["b_enc"], k_row, seed=5, p=p)
    rec = pk.read_info(info)[0]
    assert int(rec["status"]) in (0, 3)   # filtered (or the plan's exact path)
    z = osae.encode(m["x"], m["w_enc"], m["b_enc"])
    _check_selection(vals.cpu().numpy().astype(np.float64), idx.cpu().numpy(), z, _tol(m), K)
    # internal consistency: the exact top-K of the GPU's own latents, bit for bit
    t = torch()
    dense = pk.sae_encode_dense(g["x"], g["w_enc"], g["b_enc"]).reshape(-1).cpu().numpy()
    order = np.lexsort((np.arange(dense.size), -dense.astype(np.float64)))[:K]
    assert np.array_equal(idx.cpu().numpy(), order)
    assert np.array_equal(vals.cpu().numpy().view(np.uint32), dense[order].view(np.uint32))


def _exact_topk_of(dense, K):
    """Indices of the K largest of a flat fp32 array under the total order
    (value descending, then index ascending), and their values."""
    d64 = dense.astype(np.float64)
    kth = np.partition(-d64, K - 1)[K - 1]            # minus the K-th largest value
    cand = np.nonzero(-d64 <= kth)[0]                  # every index with a value >= it
    order = cand[np.lexsort((cand, -d64[cand]))][:K]
    return order, dense[order]


@pytest.mark.parametrize("B,d_model,d_dict,k_row", [(4096, 128, 8192, 8), (4000, 192, 8000, 8), (4096, 64, 8192, 8)])
def test_sae_encode_topk_several_tiles_per_workgroup(B, d_model, d_dict, k_row):
    # more 256 x 256 filter tiles than workgroups: the next tile's loads
    # overlap an epilogue, and a tile's survivors are appended during the
    # next tile (an even d_model / 64), or each tile loads behind its own
    # barrier (odd: 3 chunks, and 1); the last row and column tiles are
    # partial in the second
    m = workloads.sae_model(B=B, d_model=d_model, d_dict=d_dict, seed=23)
    g = _dev(m)
    K = B * k_row
    p = pk.plan_sae(B, d_dict, k_row)
    note(f"sae topk tiles B={B} d_model={d_model} d_dict={d_dict} K={K} S={p.S} t={p.t} M={p.M} mode={p.mode}")
    vals, idx, info = pk.sae_encode_topk(g["x"], g["w_enc"], g["b_enc"], k_row, seed=3, p=p)
    assert int(pk.read_info(info)[0]["status"]) == 0
    dense = pk.sae_encode_dense(g["x"], g["w_enc"], g["b_enc"]).reshape(-1).cpu().numpy()
    order, ov = _exact_topk_of(dense, K)
    assert np.array_equal(idx.cpu().numpy(), order)
    assert np.array_equal(vals.cpu().numpy().view(np.uint32), ov.view(np.uint32))


def test_sae_encode_topk_default_plan():
    # the binding's default plan (profk_default_sae_opts: the sample floor)
    B, d_model, d_dict, k_row = 512, 256, 4096, 16
    m = workloads.sae_model(B=B, d_model=d_model, d_dict=d_dict, seed=19)
    g = _dev(m)
    p = pk.plan_sae(B, d_dict, k_row)
    note(f"sae default plan S={p.S} t={p.t} M={p.M} mode={p.mode}")
    vals, idx, info = pk.sae_encode_topk(g["x"], g["w_enc"], g["b_enc"], k_row, seed=1)
    assert int(pk.read_info(info)[0]["status"]) in (0, 3)
    z = osae.encode(m["x"], m["w_enc"], m["b_enc"])
    _check_selection(vals.cpu().numpy().astype(np.float64), idx.cpu().numpy(), z, _tol(m), B * k_row)


def test_sae_encode_topk_fallback():
    # a 64-draw sample with a small buffer overflows: the dense latents are
    # written to the workspace and selected exactly
    B, d_model, d_dict, k_row = 128, 128, 512, 8
    m = workloads.sae_model(B=B, d_model=d_model, d_dict=d_dict, seed=13)
    g = _dev(m)
    K = B * k_row
    p = pk.plan(B * d_dict, K, 1e-6, 1.0, S_min=64, S_max=64, force_mode=pk.FORCE_FILTER)
    p.M = K   # too small for the survivors of a 64-draw threshold
    note(f"sae fallback K={K} S={p.S} t={p.t} M={p.M}")
    vals, idx, info = pk.sae_encode_topk(g["x"], g["w_enc"], g["b_enc"], k_row, seed=2, p=p)
    rec = pk.read_info(info)[0]
    assert int(rec["status"]) in (1, 2)
    z = osae.encode(m["x"], m["w_enc"], m["b_enc"])
    _check_selection(vals.cpu().numpy().astype(np.float64), idx.cpu().numpy(), z, _tol(m), K)


@pytest.mark.parametrize("B,d_model,d_dict,k_row", [(64, 512, 2048, 32), (37, 96, 300, 5)])
def test_sae_decode(B, d_model, d_dict, k_row):
    t = torch()
    m = workloads.sae_model(B=B, d_model=d_model, d_dict=d_dict, seed=17)
    z = osae.encode(m["x"], m["w_enc"], m["b_enc"])
    K = B * k_row
    v64, i64 = osae.batchtopk(z, K)
    v32 = v64.astype(np.float32)
    # padding and a shuffled order must not change the result
    perm = np.random.default_rng(0).permutation(K)
    vals = np.r_[v32[perm], np.float32(-np.inf), np.float32(5.0)]
    idx = np.r_[i64[perm], -1, B * d_dict + 3].astype(np.int64)
    note(f"sae decode B={B} d_model={d_model} d_dict={d_dict} K={K}")
    g = _dev(m)
    out = pk.sae_decode(t.from_numpy(vals).cuda(), t.from_numpy(idx).cuda(), g["w_dec"], g["b_dec"], B)
    ref = osae.decode(v32, i64, m["w_dec"], m["b_dec"], B)
    scale = osae.decode_scale(v32, i64, m["w_dec"], m["b_dec"], B)
    per_row = np.bincount(i64 // d_dict, minlength=B)
    tol = ((per_row + 2) * U)[:, None] * scale
    got = out.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(got - ref) <= tol)
    # the same entries in the oracle's order give the same bits
    out2 = pk.sae_decode(t.from_numpy(v32).cuda(), t.from_numpy(i64).cuda(), g["w_dec"], g["b_dec"], B)
    assert t.equal(out.view(t.int32), out2.view(t.int32))
