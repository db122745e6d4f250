"""Student input features and delayed targets (§II-B).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Features: 64-dimensional log mel energies every 10 ms are stacked three at
a time and sub-sampled to a 30 ms advance, at one of three offsets per
utterance; a causal mean estimate is subtracted; then global mean and
variance normalisation is applied.  Targets: the model has a three-frame
look-ahead, so its output at frame t is scored against the target of frame
t - 3.

Readings (the paper gives the recipe in prose only):
  * stacked frame t of offset o is [F(o + 3t), F(o + 3t + 1), F(o + 3t + 2)]
    (oldest first); only complete stacks are formed, so an utterance of U
    raw frames gives max(0, (U - o - stack) // skip + 1) frames;
  * the causal mean estimate at stacked frame t is the mean of the stacked
    frames 0..t of the utterance (the frame itself included);
  * global normalisation is (z - mean) / std per dimension, with the
    statistics supplied by the caller;
  * with delay d, output row (t, b) takes the target of (t - d, b); rows with
    t < d carry no target (mask 0).  The caller extends an utterance by d
    frames if its last d targets are to be scored.
Arithmetic: fp64.
"""

import numpy as np


def lfr_frames(U, stack=3, skip=3, offset=0):
    """Stacked frames of an utterance of U raw frames."""
    return max(0, (U - offset - stack) // skip + 1)


def lfr_stack(raw, stack=3, skip=3, offset=0):
    """raw [U][D] -> stacked [T][stack * D]."""
    raw = np.asarray(raw, dtype=np.float64)
    U, D = raw.shape
    T = lfr_frames(U, stack, skip, offset)
    out = np.empty((T, stack * D))
    for t in range(T):
        for k in range(stack):
            out[t, k * D:(k + 1) * D] = raw[offset + skip * t + k]
    return out


def causal_mean_subtract(y):
    """z_t = y_t - mean(y_0 .. y_t)."""
    y = np.asarray(y, dtype=np.float64)
    run = np.zeros(y.shape[1])
    z = np.empty_like(y)
    for t in range(y.shape[0]):
        run = run + y[t]
        z[t] = y[t] - run / (t + 1)
    return z


def global_mvn(z, mean, std):
    return (np.asarray(z, np.float64) - np.asarray(mean, np.float64)) / np.asarray(std, np.float64)


def lfr_features(raw, mean, std, stack=3, skip=3, offset=0):
    """One utterance's student input frames [T][stack * D]."""
    return global_mvn(causal_mean_subtract(lfr_stack(raw, stack, skip, offset)), mean, std)


def delay_targets(idx, prob, T, B, lengths, delay):
    """Targets of the packed rows shifted by `delay` frames within each
    sequence.  idx [N][K] int32, prob [N][K]; rows in the packed time-major
    layout of the model (frame (t, b) is row off_t + b).  Returns (idx_d,
    prob_d, mask) with idx -1, prob 0 and mask 0 where t < delay."""
    from .lstm_am import batch_schedule
    counts, offs = batch_schedule(T, B, lengths)
    idx = np.asarray(idx)
    prob = np.asarray(prob)
    N, K = idx.shape
    idx_d = np.full((N, K), -1, dtype=np.int32)
    prob_d = np.zeros((N, K), dtype=prob.dtype)
    mask = np.zeros(N, dtype=np.uint8)
    for t in range(T):
        for b in range(int(counts[t])):
            row = int(offs[t]) + b
            if t >= delay:
                src = int(offs[t - delay]) + b
                idx_d[row] = idx[src]
                prob_d[row] = prob[src]
                mask[row] = 1
    return idx_d, prob_d, mask
