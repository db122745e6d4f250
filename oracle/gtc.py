"""Gradient Threshold Compression, encode and decode (fp32, exact order).

§VI-A: instead of the whole gradient, a worker sends only the elements whose
magnitude exceeds a gradient threshold tau; what is not sent stays in a local
residual and is added to later gradients.  Updates are quantised to one bit,
so every sent element means +tau or -tau, and the sign is packed with the
element index into one 32-bit word.

Readings taken here (the paper describes the rule in prose only):
  * the residual absorbs the current gradient before the test:  a = r + g;
  * the test is strict:  a > tau emits +tau,  a < -tau emits -tau;
  * one quantum per element per call; the sent quantum is removed from the
    residual (r = a - tau or a + tau) and any excess stays in it;
  * word = (flat_index << 1) | sign, sign 1 meaning -tau; words are listed in
    ascending index order, so the output is unique;
  * NaN compares false and is never sent (the residual stays NaN); +-Inf is
    sent and stays in the residual.
All arithmetic is a single fp32 add or subtract, rounded to nearest even with
IEEE subnormals; no fused operations.
"""

import numpy as np


def grad_threshold_encode(grad, residual, tau):
    """Returns (new_residual fp32 [n], words uint32 [count], count)."""
    g = np.asarray(grad, dtype=np.float32)
    r = np.asarray(residual, dtype=np.float32)
    assert g.shape == r.shape and g.ndim == 1
    assert g.shape[0] < 2 ** 31
    tau = np.float32(tau)
    a = r + g
    pos = a > tau
    neg = a < -tau
    new_r = a.copy()
    new_r[pos] = a[pos] - tau
    new_r[neg] = a[neg] + tau
    sent = np.flatnonzero(pos | neg)                 # ascending
    words = (sent.astype(np.uint32) << np.uint32(1)) | neg[sent].astype(np.uint32)
    return new_r, words, int(sent.shape[0])


def grad_threshold_decode(words, count, tau, n, dense=None, accumulate=False):
    """Dense update from ``count`` words.

    accumulate=False: the result is +-tau at every sent index, 0 elsewhere.
    accumulate=True : ``dense`` plus +-tau at every sent index (one fp32 add
    per word; one stream holds each index at most once).
    """
    tau = np.float32(tau)
    w = np.asarray(words, dtype=np.uint32)[:count]
    index = (w >> np.uint32(1)).astype(np.int64)
    value = np.where((w & np.uint32(1)) != 0, -tau, tau).astype(np.float32)
    assert np.all(index < n)
    if accumulate:
        out = np.array(dense, dtype=np.float32, copy=True)
        assert out.shape == (n,)
        np.add.at(out, index, value)
    else:
        out = np.zeros(n, dtype=np.float32)
        out[index] = value
    return out


def grad_threshold_decode_multi(words, counts, tau, n, dense=None, accumulate=False):
    """Aggregate of the sparse updates of several workers (§VI-A: every worker
    receives all sparse updates and aggregates them).

    words  [S][capacity] uint32, one encode output per worker
    counts [S]: number of valid words in each row
    The aggregate of element i is tau times the integer sum k_i of the signs
    (+1, or -1 for sign bit 1) of all words that name i, so it does not depend
    on the order of the workers.  Reading: it is evaluated as the exact product
    tau * k_i rounded once to fp32.
    accumulate=False: dense[i] = fl32(tau * k_i) where some word names i, +0.0
    elsewhere.  accumulate=True: dense[i] = fl32(dense[i] + fl32(tau * k_i))
    where some word names i, unchanged elsewhere.
    """
    tau = np.float32(tau)
    w = np.asarray(words, dtype=np.uint32)
    if w.ndim == 1:
        w = w[None, :]
    k = np.zeros(n, dtype=np.int64)
    hit = np.zeros(n, dtype=bool)
    for s in range(w.shape[0]):
        ws = w[s, :int(counts[s])]
        index = (ws >> np.uint32(1)).astype(np.int64)
        assert np.all(index < n)
        sign = np.where((ws & np.uint32(1)) != 0, -1, 1)
        np.add.at(k, index, sign)
        hit[index] = True
    v = (np.float64(tau) * k.astype(np.float64)).astype(np.float32)
    if accumulate:
        out = np.array(dense, dtype=np.float32, copy=True)
        assert out.shape == (n,)
        out[hit] = out[hit] + v[hit]
    else:
        out = np.zeros(n, dtype=np.float32)
        out[hit] = v[hit]
    return out
