"""Student-teacher cross-entropy against sparse k-best teacher targets (fp64).

§II-C and §V-A: the student is trained by minimising the cross-entropy between
the teacher's and the student's senone posteriors, the teacher being frozen.
§V-C: only the teacher's k best entries per frame are kept; the rest of the
posterior is treated as (numerically) zero.

Reading taken here: each frame f carries k (index, probability) pairs as given
(no renormalisation; their mass M_f may be below one), slots with index -1 are
empty, repeated indices add.  With the student's log-softmax
log q_fc = z_fc - lse_f, lse_f = log sum_c exp(z_fc):

    loss_f = - sum_j p_fj * log q_{f, idx_fj}
    dloss_f / dz_fc = M_f * q_fc - sum_{j: idx_fj = c} p_fj

Reduction: mean over valid frames (the sum of the mask), or a plain sum.
Each frame's term is scaled by s_f = m_f / N_valid (or m_f); a frame with mask
0 contributes nothing and gets a zero gradient row.
"""

import numpy as np

MEAN_VALID = 0
SUM = 1


def sparse_soft_ce(logits, idx, prob, mask=None, reduction=MEAN_VALID):
    """Returns (loss: float, dlogits [N][C] fp64)."""
    z = np.asarray(logits, dtype=np.float64)
    idx = np.asarray(idx, dtype=np.int64)
    p = np.asarray(prob, dtype=np.float64)
    N, C = z.shape
    assert idx.shape == p.shape and idx.shape[0] == N
    assert np.all((idx >= -1) & (idx < C))
    m = np.ones(N) if mask is None else (np.asarray(mask) != 0).astype(np.float64)

    if reduction == MEAN_VALID:
        nv = m.sum()
        scale = m / nv if nv > 0 else np.zeros(N)
    elif reduction == SUM:
        scale = m
    else:
        raise ValueError("unknown reduction")

    loss = 0.0
    dz = np.zeros((N, C))
    for f in range(N):
        if scale[f] == 0.0:
            continue
        zmax = z[f].max()
        lse = zmax + np.log(np.exp(z[f] - zmax).sum())
        q = np.exp(z[f] - lse)
        mass = 0.0
        lf = 0.0
        target = np.zeros(C)
        for j in range(idx.shape[1]):
            c = idx[f, j]
            if c < 0:
                continue
            mass += p[f, j]
            lf -= p[f, j] * (z[f, c] - lse)
            target[c] += p[f, j]
        loss += scale[f] * lf
        dz[f] = scale[f] * (mass * q - target)
    return loss, dz
