"""Seeded synthetic inputs shaped like the paper's student-training workloads.

This module only draws random numbers; it holds none of the training step's
arithmetic and is shared by the tests, the benchmark and the oracle checks.

Stand-ins for data the paper trains on (Alexa production speech, not public):
  * features: 192-dim frames (64 log-mel energies stacked 3 at a time, §II-B)
    after global mean/variance normalisation (§IV-B), modelled as i.i.d. N(0,1);
  * teacher targets: the k best senones per frame (§V-C, k = 20 in §VII),
    indices drawn without replacement from a Zipf(1.1) law over the senones,
    probabilities from a symmetric Dirichlet(0.3) scaled to the stated mass;
  * chunks: fixed-length chunks for chunked BPTT (§II-B) or whole utterances of
    varying length, sorted longest first.

Stand-ins for the state of several data-parallel workers (one GPU plays all
of them): local models that drifted from the global model over a block of
local SGD (the global model plus N(0, spread^2) noise per worker), and
per-worker gradients of the scale of the training step's (N(0, scale^2)).

Stand-in for raw 10 ms log mel energies (before stacking, §II-B): per
utterance a per-dimension level N(2, 3^2) plus a slow random-walk drift
(so that the causal mean matters) plus N(0, 1) frame noise.

Seeds: weights 0, features 1, targets 2, lengths 3, one-hot frame choice 4,
worker models 5, worker gradients 6, raw log mel frames 7.
"""

import numpy as np

SEED_WEIGHTS, SEED_FEATURES, SEED_TARGETS, SEED_LENGTHS, SEED_ONEHOT = 0, 1, 2, 3, 4
SEED_WORKER_MODELS, SEED_WORKER_GRADS, SEED_RAW = 5, 6, 7

# Workload shapes.  dtype "f32": fp32 throughout; "bf16": bf16 weights and
# activations with fp32 master weights.
WORKLOADS = {
    "tiny-2x64": dict(layers=2, input_dim=64, hidden=64, classes=500,
                      T=50, B=16, K=5, mass=0.95, dtype="f32", lr=0.01, tau=1e-3),
    "paper-5x768": dict(layers=5, input_dim=192, hidden=768, classes=3000,
                        T=64, B=256, K=20, mass=0.98, dtype="bf16", lr=0.01, tau=1e-4),
    "wide-5x1536": dict(layers=5, input_dim=192, hidden=1536, classes=6000,
                        T=64, B=512, K=20, mass=0.98, dtype="bf16", lr=0.01, tau=1e-4),
    "varlen-5x768": dict(layers=5, input_dim=192, hidden=768, classes=3000,
                         T=1500, B=128, K=20, mass=0.98, dtype="bf16", lr=0.01, tau=1e-4,
                         len_lo=200, len_hi=1500, one_hot_frac=0.1),
}


def init_params(n, hidden, seed=SEED_WEIGHTS):
    """fp32 master weights, every entry U(-1/sqrt(H), 1/sqrt(H))."""
    rng = np.random.default_rng(seed)
    bound = 1.0 / np.sqrt(hidden)
    return rng.uniform(-bound, bound, size=n).astype(np.float32)


def features(n_frames, dim, seed=SEED_FEATURES):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((n_frames, dim), dtype=np.float32)


def utterance_lengths(batch, lo, hi, seed=SEED_LENGTHS):
    """Lengths uniform on {lo..hi}, sorted non-increasing."""
    rng = np.random.default_rng(seed)
    lens = rng.integers(lo, hi + 1, size=batch)
    return np.sort(lens)[::-1].astype(np.int32).copy()


def teacher_targets(n_frames, classes, k, mass, seed=SEED_TARGETS, zipf_s=1.1,
                    alpha=0.3, one_hot_frac=0.0, seed_onehot=SEED_ONEHOT,
                    chunk=1024):
    """Sparse teacher posteriors: idx int32 [N][k] (-1 = empty slot), prob fp32.

    Zipf draws without replacement use the Gumbel-top-k construction (the k
    largest of log p_c + Gumbel noise are a sample without replacement,
    listed in draw order).  With ``one_hot_frac`` > 0, that fraction of frames
    (Bernoulli, own seed) keeps only its first drawn index, with probability
    1.0, and marks the other slots empty.
    """
    rng = np.random.default_rng(seed)
    logp = -zipf_s * np.log(np.arange(1, classes + 1, dtype=np.float64))
    idx = np.empty((n_frames, k), dtype=np.int32)
    for s in range(0, n_frames, chunk):
        e = min(n_frames, s + chunk)
        keys = logp[None, :] + rng.gumbel(size=(e - s, classes))
        part = np.argpartition(-keys, k - 1, axis=1)[:, :k]
        order = np.argsort(-np.take_along_axis(keys, part, axis=1), axis=1)
        idx[s:e] = np.take_along_axis(part, order, axis=1)
    prob = (mass * rng.dirichlet(np.full(k, alpha), size=n_frames)).astype(np.float32)
    if one_hot_frac > 0.0:
        sel = np.random.default_rng(seed_onehot).random(n_frames) < one_hot_frac
        idx[sel, 1:] = -1
        prob[sel, 0] = 1.0
        prob[sel, 1:] = 0.0
    return idx, prob


def worker_models(base, workers, spread, seed=SEED_WORKER_MODELS):
    """[workers][n] fp32: base plus independent N(0, spread^2) drift per worker."""
    rng = np.random.default_rng(seed)
    base = np.asarray(base, dtype=np.float32)
    out = np.empty((workers, base.shape[0]), dtype=np.float32)
    for i in range(workers):
        out[i] = base + (rng.standard_normal(base.shape[0], dtype=np.float32) * np.float32(spread))
    return out


def worker_gradients(n, workers, scale, seed=SEED_WORKER_GRADS):
    """[workers][n] fp32 gradients, i.i.d. N(0, scale^2)."""
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((workers, n), dtype=np.float32) * np.float32(scale))


def raw_logmel(raw_lengths, dim=64, seed=SEED_RAW):
    """[sum raw_lengths][dim] fp32, utterance after utterance."""
    rng = np.random.default_rng(seed)
    parts = []
    for U in raw_lengths:
        level = rng.normal(2.0, 3.0, dim)
        drift = np.cumsum(rng.normal(0.0, 0.05, (int(U), dim)), axis=0)
        parts.append(level[None, :] + drift + rng.standard_normal((int(U), dim)))
    if not parts:
        return np.zeros((0, dim), np.float32)
    return np.concatenate(parts).astype(np.float32)
