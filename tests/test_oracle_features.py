"""Pins of the oracle's input features and delayed targets (§II-B): the
stacked layout on frames that encode their own position, frame counts per
offset, a closed form of the causal mean on a ramp, the statistics after
global normalisation, the delayed targets on targets that encode their own
(sequence, frame), the delayed loss against slices aligned by hand, and a
chunked forward with carried state against the unchunked one.  CPU only."""

import numpy as np
import pytest

import oracle
from oracle import ModelDims, param_count


@pytest.mark.parametrize("offset", [0, 1, 2])
def test_stacked_layout(offset):
    U, D = 20, 64
    raw = 1000.0 * np.arange(U)[:, None] + np.arange(D)[None, :]
    y = oracle.lfr_stack(raw, 3, 3, offset)
    assert y.shape == (oracle.lfr_frames(U, 3, 3, offset), 3 * D)
    for t in range(y.shape[0]):
        for k in range(3):
            np.testing.assert_array_equal(y[t, k * D:(k + 1) * D], 1000.0 * (offset + 3 * t + k) + np.arange(D))


@pytest.mark.parametrize("U,offset,T", [(0, 0, 0), (2, 0, 0), (3, 0, 1), (5, 0, 1), (6, 0, 2), (9, 0, 3),
                                        (4, 1, 1), (4, 2, 0), (5, 2, 1), (100, 1, 33), (100, 2, 32)])
def test_frame_counts(U, offset, T):
    assert oracle.lfr_frames(U, 3, 3, offset) == T


def test_offsets_cover_every_raw_frame():
    U = 31
    used = set()
    for o in range(3):
        for t in range(oracle.lfr_frames(U, 3, 3, o)):
            used.add(o + 3 * t)  # each stack starts at a distinct raw frame
    assert used == set(range(U - 2))


def test_causal_mean_closed_forms():
    T, D = 50, 7
    const = np.full((T, D), 3.25)
    np.testing.assert_allclose(oracle.causal_mean_subtract(const), 0.0, atol=1e-13)
    a, b = np.linspace(-1, 1, D), np.linspace(0.5, 2, D)
    ramp = a[None, :] + b[None, :] * np.arange(T)[:, None]
    # mean of a + b s over s <= t is a + b t / 2, so z_t = b t / 2
    np.testing.assert_allclose(oracle.causal_mean_subtract(ramp), b[None, :] * np.arange(T)[:, None] / 2,
                               rtol=1e-12, atol=1e-12)
    rnd = np.random.default_rng(0).standard_normal((T, D))
    np.testing.assert_array_equal(oracle.causal_mean_subtract(rnd)[0], 0.0)


def test_global_normalisation_statistics():
    rng = np.random.default_rng(1)
    z = rng.standard_normal((20000, 5)) * np.array([1, 2, 3, 4, 5]) + np.array([5, 4, 3, 2, 1])
    out = oracle.global_mvn(z, z.mean(axis=0), z.std(axis=0))
    np.testing.assert_allclose(out.mean(axis=0), 0.0, atol=1e-12)
    np.testing.assert_allclose(out.std(axis=0), 1.0, rtol=1e-12)


def _packed(T, B, lengths, K):
    """Targets whose idx encodes (sequence, frame) as 1000 b + t, in the
    packed layout, built sequence by sequence."""
    rows = []
    for t in range(T):
        for b in range(B):
            if lengths is None or lengths[b] > t:
                rows.append((b, t))
    idx = np.array([[1000 * b + t] * K for b, t in rows], np.int32)
    prob = np.array([[0.1 * (k + 1)] * 1 for k in range(K)], np.float32).T.repeat(len(rows), 0)
    return idx, prob, rows


@pytest.mark.parametrize("lengths", [None, [9, 7, 7, 3, 2, 0]])
@pytest.mark.parametrize("delay", [0, 1, 3])
def test_delayed_targets(lengths, delay):
    T, B, K = 9, 6, 4
    idx, prob, rows = _packed(T, B, lengths, K)
    idx_d, prob_d, mask = oracle.delay_targets(idx, prob, T, B, lengths, delay)
    for r, (b, t) in enumerate(rows):
        if t < delay:
            assert mask[r] == 0 and np.all(idx_d[r] == -1) and np.all(prob_d[r] == 0)
        else:
            assert mask[r] == 1
            assert np.all(idx_d[r] == 1000 * b + (t - delay))
            np.testing.assert_array_equal(prob_d[r], prob[r])


def test_delayed_loss_equals_aligned_slices():
    T, B, C, K, d = 10, 4, 30, 5, 3
    rng = np.random.default_rng(2)
    logits = rng.standard_normal((T * B, C))
    idx = np.stack([rng.permutation(C)[:K] for _ in range(T * B)]).astype(np.int32)
    prob = (0.9 * rng.dirichlet(np.ones(K), T * B)).astype(np.float32)
    idx_d, prob_d, mask = oracle.delay_targets(idx, prob, T, B, None, d)
    loss, dz = oracle.sparse_soft_ce(logits, idx_d, prob_d, mask)
    # by hand: outputs of frames d.. against targets of frames 0..T-d-1
    L3 = logits.reshape(T, B, C)[d:].reshape(-1, C)
    ref_loss, ref_dz = oracle.sparse_soft_ce(L3, idx.reshape(T, B, K)[:T - d].reshape(-1, K),
                                            prob.reshape(T, B, K)[:T - d].reshape(-1, K))
    assert loss == pytest.approx(ref_loss, rel=1e-12)
    np.testing.assert_allclose(dz.reshape(T, B, C)[d:].reshape(-1, C), ref_dz, rtol=1e-12, atol=1e-15)
    np.testing.assert_array_equal(dz.reshape(T, B, C)[:d], 0.0)


def test_chunked_forward_with_carried_state_equals_unchunked():
    dims = ModelDims(2, 6, 8, 11)
    T, B = 12, 3
    rng = np.random.default_rng(3)
    p = rng.uniform(-0.4, 0.4, param_count(dims))
    x = rng.standard_normal((T * B, dims.input_dim))
    full, cache = oracle.lstm_am_forward(p, dims, x, T, B)
    a, ca = oracle.lstm_am_forward(p, dims, x[:5 * B], 5, B)
    b, cb = oracle.lstm_am_forward(p, dims, x[5 * B:], T - 5, B, None, ca["hT"], ca["cT"])
    np.testing.assert_array_equal(np.concatenate([a, b]), full)
    np.testing.assert_array_equal(cb["hT"], cache["hT"])
    np.testing.assert_array_equal(cb["cT"], cache["cT"])
