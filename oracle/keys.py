"""Order-preserving keys: the total order every result is defined under.

Test infrastructure (see the package docstring).  The paper asks for "the k
largest entries together with their indices" (Sec. 3, problem statement) and
says nothing about ties, signed zeros or NaN.  The reading used here:

  key(x) is the IEEE bit pattern u of x with every bit flipped when the sign
  bit is set, and only the sign bit set otherwise.  Comparing keys as unsigned
  integers then orders -NaN < -inf < ... < -0.0 < +0.0 < ... < +inf < +NaN.

  Element i precedes element j iff key_i > key_j, or key_i == key_j and i < j.

Arrays of bf16 values are carried as their uint16 bit patterns (numpy has no
bf16 type); the same rule applies on 16 bits.
"""

import numpy as np


def f32_bits(x):
    """Bit patterns (uint32) of a float32 array."""
    return np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)


def key_u32(bits):
    """Key of fp32 bit patterns: flip all bits of negatives, set the sign bit
    of non-negatives."""
    u = np.asarray(bits, dtype=np.uint32)
    negative = (u >> np.uint32(31)) == 1
    return np.where(negative, ~u, u | np.uint32(0x80000000)).astype(np.uint32)


def key_u16(bits):
    """Key of bf16 bit patterns (uint16), same rule on 16 bits."""
    u = np.asarray(bits, dtype=np.uint16)
    negative = (u >> np.uint16(15)) == 1
    return np.where(negative, ~u, u | np.uint16(0x8000)).astype(np.uint16)


def bits_from_key_u32(key):
    """Inverse of key_u32."""
    kk = np.asarray(key, dtype=np.uint32)
    was_nonneg = (kk >> np.uint32(31)) == 1
    return np.where(was_nonneg, kk & np.uint32(0x7FFFFFFF), ~kk).astype(np.uint32)


def bits_from_key_u16(key):
    """Inverse of key_u16."""
    kk = np.asarray(key, dtype=np.uint16)
    was_nonneg = (kk >> np.uint16(15)) == 1
    return np.where(was_nonneg, kk & np.uint16(0x7FFF), ~kk).astype(np.uint16)


def keys_of(bits, dtype):
    """Keys of a bit-pattern array; dtype is 'f32' (uint32 bits) or 'bf16'
    (uint16 bits).  Keys come back as int64 so both widths compare alike."""
    if dtype == "f32":
        return key_u32(bits).astype(np.int64)
    if dtype == "bf16":
        return key_u16(bits).astype(np.int64)
    raise ValueError(f"unknown dtype {dtype!r}")
