"""Pins for O3 (oracle.sae): the SAE layer around the BatchTopK selection.

Checks closed forms (identity and one-hot encoders, single-entry decodes),
brute-force loops on tiny cases, known bf16 bit patterns, and invariants
(linearity of the decode, the error scale bounding every sum)."""

import math

import numpy as np
import pytest

from oracle import sae
import workloads


def _bits(a):
    return workloads.f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


def test_bf16_bit_patterns():
    bits = np.array([0x3F80, 0xC000, 0x0000, 0x8000, 0x7F80, 0x3E80, 0x4049], dtype=np.uint16)
    v = sae.bf16_to_f64(bits)
    assert list(v[:4]) == [1.0, -2.0, 0.0, 0.0] and math.copysign(1.0, v[3]) == -1.0
    assert math.isinf(v[4]) and v[5] == 0.25 and v[6] == 3.140625


def test_identity_encoder_is_relu_of_x_plus_bias():
    g = np.random.default_rng(0)
    x = _bits(g.standard_normal((5, 16)))
    b = g.standard_normal(16).astype(np.float32)
    eye = _bits(np.eye(16))
    z = sae.encode(x, eye, b)
    xv = sae.bf16_to_f64(x)
    for r in range(5):
        for j in range(16):
            assert z[r, j] == max(xv[r, j] + float(b[j]), 0.0)


def test_one_hot_encoder_rows_gather_scaled_inputs():
    g = np.random.default_rng(1)
    d_model, d_dict = 8, 12
    perm = g.integers(0, d_model, d_dict)
    scale = np.array([2.0, -0.5, 4.0, 1.0, -1.0, 0.25, 8.0, -2.0, 0.5, 3.0, -4.0, 1.5])
    w = np.zeros((d_dict, d_model), dtype=np.float32)
    w[np.arange(d_dict), perm] = scale
    x = _bits(g.standard_normal((3, d_model)))
    b = np.zeros(d_dict, dtype=np.float32)
    z = sae.encode(x, _bits(w), b)
    xv = sae.bf16_to_f64(x)
    for r in range(3):
        for j in range(d_dict):
            assert z[r, j] == max(scale[j] * xv[r, perm[j]], 0.0)


def test_encode_matches_loops_on_a_tiny_layer():
    m = workloads.sae_model(B=3, d_model=7, d_dict=5, seed=2)
    z = sae.encode(m["x"], m["w_enc"], m["b_enc"])
    s = sae.encode_scale(m["x"], m["w_enc"], m["b_enc"])
    xv, wv = sae.bf16_to_f64(m["x"]), sae.bf16_to_f64(m["w_enc"])
    for r in range(3):
        for j in range(5):
            acc = float(m["b_enc"][j])
            mag = abs(float(m["b_enc"][j]))
            for c in range(7):
                acc += xv[r, c] * wv[j, c]
                mag += abs(xv[r, c] * wv[j, c])
            assert z[r, j] == pytest.approx(max(acc, 0.0), rel=1e-15, abs=1e-15)
            assert s[r, j] == pytest.approx(mag, rel=1e-15)
            assert abs(acc) <= s[r, j] * (1 + 1e-12)


def test_batchtopk_is_the_sorted_prefix_with_ties_by_index():
    z = np.array([[0.0, 3.0, 1.0, 3.0], [2.0, 0.0, 3.0, 1.0]])
    v, i = sae.batchtopk(z, 5)
    brute = sorted(range(8), key=lambda f: (-z.reshape(-1)[f], f))[:5]
    assert list(i) == brute == [1, 3, 6, 4, 2]
    assert list(v) == [3.0, 3.0, 3.0, 2.0, 1.0]


def test_decode_of_one_entry_per_row():
    m = workloads.sae_model(B=4, d_model=6, d_dict=9, seed=3)
    vals = np.array([1.5, 0.25, 2.0, 3.0])
    idx = np.array([0 * 9 + 4, 1 * 9 + 0, 2 * 9 + 8, 3 * 9 + 4], dtype=np.int64)
    out = sae.decode(vals, idx, m["w_dec"], m["b_dec"], 4)
    w = sae.bf16_to_f64(m["w_dec"])
    for r, (v, f) in enumerate(zip(vals, idx)):
        j = int(f) % 9
        assert np.array_equal(out[r], v * w[j] + m["b_dec"].astype(np.float64))


def test_decode_is_linear_and_skips_padding():
    m = workloads.sae_model(B=3, d_model=5, d_dict=7, seed=4)
    g = np.random.default_rng(5)
    i1 = g.choice(21, 6, replace=False)
    i2 = np.setdiff1d(np.arange(21), i1)[:6]
    v1, v2 = g.random(6), g.random(6)
    b0 = sae.decode([], [], m["w_dec"], m["b_dec"], 3)
    both = sae.decode(np.r_[v1, v2, 9.0], np.r_[i1, i2, -1], m["w_dec"], m["b_dec"], 3)
    parts = sae.decode(v1, i1, m["w_dec"], m["b_dec"], 3) + sae.decode(v2, i2, m["w_dec"], m["b_dec"], 3) - b0
    assert np.allclose(both, parts, rtol=0, atol=1e-12)
    assert np.array_equal(b0, np.tile(m["b_dec"].astype(np.float64), (3, 1)))
    s = sae.decode_scale(np.r_[v1, v2], np.r_[i1, i2], m["w_dec"], m["b_dec"], 3)
    assert np.all(np.abs(both) <= s * (1 + 1e-12))


def test_decode_scale_matches_loops_on_a_tiny_layer():
    """decode_scale written out: for each row, sum over its selected
    latents of |v| |W_dec[j, c]|, plus |b_dec[c]|.  Values and weights of
    both signs, a padding entry, and a row with no latent."""
    B, d_model, d_dict = 4, 6, 9
    m = workloads.sae_model(B=B, d_model=d_model, d_dict=d_dict, seed=7)
    g = np.random.default_rng(8)
    idx = np.array([0 * 9 + 2, 0 * 9 + 7, 1 * 9 + 0, 2 * 9 + 5, 2 * 9 + 1, 2 * 9 + 8, -1], dtype=np.int64)
    vals = g.standard_normal(idx.size) * 3.0
    b_dec = g.standard_normal(d_model).astype(np.float32)
    w = sae.bf16_to_f64(m["w_dec"])
    assert (w < 0).any() and (vals < 0).any() and (b_dec < 0).any()
    s = sae.decode_scale(vals, idx, m["w_dec"], b_dec, B)
    for r in range(B):
        for c in range(d_model):
            mag = abs(float(b_dec[c]))
            for v, f in zip(vals, idx):
                if f < 0 or int(f) // d_dict != r:
                    continue
                mag += abs(v) * abs(w[int(f) % d_dict, c])
            assert s[r, c] == pytest.approx(mag, rel=1e-15, abs=0.0), (r, c)
    # row 3 holds no latent: only the bias magnitude
    assert np.array_equal(s[3], np.abs(b_dec.astype(np.float64)))
