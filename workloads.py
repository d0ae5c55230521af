"""Seeded synthetic inputs shaped like the Prof-K evaluation workloads.

These generators hold none of the method's arithmetic; they only produce
input arrays (fp32 as float32 arrays, bf16 as uint16 bit patterns) that both
the HIP library and the CPU oracle consume.  Shapes and value distributions
follow the paper's synthetic study (Sec. 5: Uniform, Standard Normal and
heavy-tailed Pareto inputs, N in [2^22, 2^30]) and the BatchTopK SAE
application (Sec. 5: a B x d_dict latent matrix flattened for a global
top-(B k)).  The SAE activations themselves are not available, so the
latent matrices are synthetic stand-ins.
"""

import numpy as np


def rng(seed):
    return np.random.default_rng(seed)


def uniform_f32(n, seed=0):
    """Uniform(0, 1) fp32."""
    return rng(seed).random(n, dtype=np.float32)


def normal_f32(n, seed=1):
    """Standard normal fp32."""
    return rng(seed).standard_normal(n, dtype=np.float32)


def pareto_f32(n, seed=2, a=1.1):
    """Pareto with shape a and scale 1 (drawn in fp64, cast to fp32)."""
    return (rng(seed).pareto(a, n) + 1.0).astype(np.float32)


def zeros90_f32(n, seed=2):
    """Exactly floor(0.9 n) entries +0.0; the rest Uniform(0,1) fp32 placed
    at distinct random positions."""
    g = rng(seed)
    n_nz = n - (9 * n) // 10
    x = np.zeros(n, dtype=np.float32)
    pos = g.choice(n, n_nz, replace=False)
    x[pos] = g.random(n_nz, dtype=np.float32)
    return x


def ramp_f32(n):
    """x_i = float32(i), ascending (round-to-nearest-even above 2^24 creates
    runs of equal values)."""
    return np.arange(n, dtype=np.int64).astype(np.float32)


def plateau_f32(n, seed=2, first_rank=257, width=10_000):
    """Uniform(0,1) fp32 where the elements at descending ranks
    first_rank .. first_rank+width-1 (1-based) all take the value found at
    rank first_rank: a plateau of `width` equal values."""
    x = rng(seed).random(n, dtype=np.float32)
    last = first_rank + width - 1
    top = np.argpartition(-x, last - 1)[:last]
    top = top[np.argsort(-x[top], kind="stable")]
    v = x[top[first_rank - 1]]
    x[top[first_rank - 1:last]] = v
    return x


def f32_to_bf16_bits(x):
    """Round-to-nearest-even fp32 -> bf16 bit patterns (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def relu_normal_bf16(shape, seed=3):
    """bf16 bits of max(N(0,1), +0.0): ReLU activations, about half zeros."""
    x = rng(seed).standard_normal(shape, dtype=np.float32)
    np.maximum(x, np.float32(0.0), out=x)
    return f32_to_bf16_bits(x)


def sae_preacts_f32(B=4096, D=65536, seed=4, hot_every=100, hot_shift=3.0):
    """BatchTopK stand-in: N(-0.5, 1) pre-activations of shape [B, D] where
    every column c with c % hot_every == 0 is shifted by +hot_shift."""
    x = rng(seed).standard_normal((B, D), dtype=np.float32)
    x -= np.float32(0.5)
    x[:, ::hot_every] += np.float32(hot_shift)
    return x


def special_f32(n, seed=5):
    """Small adversarial vector for edge tests: ties, signed zeros,
    infinities and NaNs of both signs mixed into a few distinct values."""
    g = rng(seed)
    pool = np.array([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, 2.5, 2.5,
                     np.nan, 3.0, 1e-38, -1e-38], dtype=np.float32)
    x = pool[g.integers(0, pool.size, n)].copy()
    u = x.view(np.uint32)
    neg_nan = g.random(n) < 0.05
    u[neg_nan] = np.uint32(0xFFC00001)
    return x


def sae_model(B=4096, d_model=512, d_dict=12288, seed=6, hot_every=100):
    """A synthetic BatchTopK SAE layer in the paper's shape (B x d_model
    inputs, d_dict latents), as bf16 bit patterns and fp32 biases:
      x      [B, d_model]       N(0, 1) activations;
      W_enc  [d_dict, d_model]  N(0, 1/d_model) rows, so pre-activations are
                                about N(0, 1);
      b_enc  [d_dict]           -0.5, and +1.5 on every hot_every-th latent
                                (frequently active latents);
      W_dec  [d_dict, d_model]  unit-norm rows;
      b_dec  [d_model]          N(0, 0.1)."""
    g = rng(seed)
    x = g.standard_normal((B, d_model), dtype=np.float32)
    w_enc = g.standard_normal((d_dict, d_model), dtype=np.float32) / np.float32(np.sqrt(d_model))
    b_enc = np.full(d_dict, -0.5, dtype=np.float32)
    b_enc[::hot_every] = np.float32(1.5)
    w_dec = g.standard_normal((d_dict, d_model), dtype=np.float32)
    w_dec /= np.linalg.norm(w_dec, axis=1, keepdims=True).astype(np.float32)
    b_dec = (g.standard_normal(d_model, dtype=np.float32) * np.float32(0.1)).astype(np.float32)
    return dict(x=f32_to_bf16_bits(x), w_enc=f32_to_bf16_bits(w_enc), b_enc=b_enc,
                w_dec=f32_to_bf16_bits(w_dec), b_dec=b_dec)
