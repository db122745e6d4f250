"""Storage-precision helpers of the oracle.

The paper does not fix a numeric precision.  The low-precision path keeps
fp32 master weights and trains from a bf16 copy; bf16 here means the upper
16 bits of an IEEE binary32 value, rounded to nearest with ties to even.
NaN maps to the canonical quiet NaN 0x7FC0; +-Inf and signed zeros are kept.
"""

import numpy as np


def bf16_bits(x):
    """fp32 -> bf16 bit patterns (uint16), round to nearest even."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    rounded = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    out = (rounded & np.uint64(0xFFFF)).astype(np.uint16)
    out[np.isnan(x)] = np.uint16(0x7FC0)
    return out


def bf16_bits_to_f32(bits):
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def bf16_round(x):
    """Value of ``x`` after a round trip through bf16, as fp32."""
    return bf16_bits_to_f32(bf16_bits(x))
