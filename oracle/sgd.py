"""Local mini-batch SGD step (§VI; each BMUF worker "updates its local model
using mini-batch SGD", §VI-B; GTC workers update from the aggregated sparse
update, §VI-A).

Plain SGD, as the paper names no momentum or weight decay for the local step:

    w <- w - lr * u

computed in fp64 from the fp32 master weight and update and rounded once to
fp32 (lr * u of two fp32 values is exact in fp64).  The bf16 working copy of
the weights is the round-to-nearest-even image of the new fp32 master.
"""

import numpy as np

from .numerics import bf16_bits


def sgd_apply(master, update, lr):
    """Returns (new fp32 master, bf16 bit patterns of it)."""
    w = np.asarray(master, dtype=np.float32).astype(np.float64)
    u = np.asarray(update, dtype=np.float32).astype(np.float64)
    lr64 = np.float64(np.float32(lr))
    new = (w - lr64 * u).astype(np.float32)
    return new, bf16_bits(new)
