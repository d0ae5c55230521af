"""O3: the BatchTopK SAE layer around the selection (Sec. 5, "Application:
BatchTopK Sparse Autoencoders").

Test infrastructure (see the package docstring).  fp64 throughout; inputs
are bf16 bit patterns (uint16) and fp32 biases, as the GPU path takes them.

The paper selects the K = B*k largest of the B x d_dict post-ReLU latents,
flattened.  The encoder that produces them is the BatchTopK SAE it builds on
(Bussmann et al.), read here as
    pre[b, j] = sum_m x[b, m] * W_enc[j, m] + b_enc[j],   z = max(pre, 0),
and the decoder as
    x_hat[b, :] = sum over selected (b, j) of z[b, j] * W_dec[j, :] + b_dec.
The exact definitions are written out below (numpy matmul as the sum); the
GPU computes the same sums in fp32 (bf16 products, one rounding per
16-product step), so comparisons use `encode_scale` to bound the rounding.
"""

import numpy as np


def bf16_to_f64(bits):
    """bf16 bit patterns -> fp64 values (exact)."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def encode(x_bits, w_enc_bits, b_enc):
    """Post-ReLU latents z [B, d_dict] in fp64."""
    pre = bf16_to_f64(x_bits) @ bf16_to_f64(w_enc_bits).T + np.asarray(b_enc, dtype=np.float64)
    return np.maximum(pre, 0.0)


def encode_scale(x_bits, w_enc_bits, b_enc):
    """sum_m |x[b,m] W_enc[j,m]| + |b_enc[j]|: the magnitude a rounded sum's
    error is proportional to."""
    return np.abs(bf16_to_f64(x_bits)) @ np.abs(bf16_to_f64(w_enc_bits)).T + \
        np.abs(np.asarray(b_enc, dtype=np.float64))


def batchtopk(z, K):
    """The K largest latents of the flattened z: (values desc, flat indices),
    ties by smaller index."""
    flat = np.asarray(z, dtype=np.float64).reshape(-1)
    order = np.lexsort((np.arange(flat.size), -flat))[:K]
    return flat[order], order.astype(np.int64)


def decode(vals, flat_idx, w_dec_bits, b_dec, B):
    """x_hat [B, d_model] from the selected latents."""
    w = bf16_to_f64(w_dec_bits)
    d_dict, d_model = w.shape
    out = np.tile(np.asarray(b_dec, dtype=np.float64), (B, 1))
    for v, i in zip(np.asarray(vals, dtype=np.float64), np.asarray(flat_idx, dtype=np.int64)):
        if i < 0:
            continue
        b, j = divmod(int(i), d_dict)
        out[b] += v * w[j]
    return out


def decode_scale(vals, flat_idx, w_dec_bits, b_dec, B):
    """sum over a row's terms of |v| |W_dec[j, :]| + |b_dec|: the error scale
    of a rounded decode."""
    sign_cleared = np.asarray(w_dec_bits, dtype=np.uint16) & np.uint16(0x7FFF)
    return decode(np.abs(vals), flat_idx, sign_cleared, np.abs(b_dec), B)
