"""Pins of the oracle's sparse soft-target cross-entropy: it must equal the
dense cross-entropy of torch when k covers every class, the textbook NLL when
k = 1, and obey the loss's invariants.  CPU only."""

import numpy as np
import pytest
import torch

import oracle
from oracle.soft_ce import MEAN_VALID, SUM


def _dense_torch(z, P):
    zt = torch.tensor(z, requires_grad=True)
    loss = torch.nn.functional.cross_entropy(zt, torch.tensor(P), reduction="mean")
    loss.backward()
    return float(loss), zt.grad.numpy()


@pytest.mark.parametrize("mass", [1.0, 0.9])
def test_k_equals_C_is_dense_cross_entropy(mass):
    rng = np.random.default_rng(0)
    N, C = 37, 23
    z = rng.standard_normal((N, C)) * 3
    P = rng.dirichlet(np.full(C, 0.5), size=N) * mass
    idx = np.stack([rng.permutation(C) for _ in range(N)])     # all classes, any order
    prob = np.take_along_axis(P, idx, axis=1)
    loss, dz = oracle.sparse_soft_ce(z, idx, prob)
    tl, tg = _dense_torch(z, P)
    assert loss == pytest.approx(tl, rel=1e-12)
    np.testing.assert_allclose(dz, tg, rtol=1e-10, atol=1e-15)


def test_k1_is_nll():
    rng = np.random.default_rng(1)
    N, C = 50, 31
    z = rng.standard_normal((N, C)) * 4
    y = rng.integers(0, C, size=N)
    loss, dz = oracle.sparse_soft_ce(z, y[:, None], np.ones((N, 1)))
    zt = torch.tensor(z, requires_grad=True)
    tl = torch.nn.functional.cross_entropy(zt, torch.tensor(y))
    tl.backward()
    assert loss == pytest.approx(float(tl), rel=1e-12)
    np.testing.assert_allclose(dz, zt.grad.numpy(), rtol=1e-10, atol=1e-15)


def _sparse_case(seed=2, N=40, C=29, K=6):
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((N, C)) * 2
    idx = np.stack([rng.choice(C, K, replace=False) for _ in range(N)])
    prob = rng.dirichlet(np.full(K, 0.3), size=N) * 0.95
    return z, idx, prob


def test_gradient_rows_sum_to_zero_and_shift_invariance():
    z, idx, prob = _sparse_case()
    loss, dz = oracle.sparse_soft_ce(z, idx, prob)
    np.testing.assert_allclose(dz.sum(axis=1), 0.0, atol=1e-15)
    shift = np.random.default_rng(3).standard_normal((z.shape[0], 1)) * 50
    loss2, dz2 = oracle.sparse_soft_ce(z + shift, idx, prob)
    assert loss2 == pytest.approx(loss, rel=1e-11)
    np.testing.assert_allclose(dz2, dz, rtol=1e-9, atol=1e-14)


def test_gradient_matches_central_differences():
    z, idx, prob = _sparse_case(N=6, C=9, K=3)
    _, dz = oracle.sparse_soft_ce(z, idx, prob)
    eps = 1e-6
    fd = np.zeros_like(z)
    for f in range(z.shape[0]):
        for c in range(z.shape[1]):
            zp = z.copy(); zp[f, c] += eps
            zm = z.copy(); zm[f, c] -= eps
            fd[f, c] = (oracle.sparse_soft_ce(zp, idx, prob)[0]
                        - oracle.sparse_soft_ce(zm, idx, prob)[0]) / (2 * eps)
    np.testing.assert_allclose(dz, fd, rtol=1e-6, atol=1e-9)


def test_mask_empty_slots_duplicates_and_sum():
    z, idx, prob = _sparse_case(N=20)
    mask = (np.arange(20) % 3 != 0).astype(np.uint8)
    loss, dz = oracle.sparse_soft_ce(z, idx, prob, mask)
    sub_loss, sub_dz = oracle.sparse_soft_ce(z[mask == 1], idx[mask == 1], prob[mask == 1])
    assert loss == pytest.approx(sub_loss, rel=1e-13)
    np.testing.assert_array_equal(dz[mask == 0], 0.0)
    np.testing.assert_allclose(dz[mask == 1], sub_dz, rtol=1e-13, atol=0)
    # empty slot (-1) contributes nothing
    idx2 = idx.copy(); prob2 = prob.copy()
    idx2[:, -1] = -1
    l_a, d_a = oracle.sparse_soft_ce(z, idx2, prob2)
    l_b, d_b = oracle.sparse_soft_ce(z, idx[:, :-1], prob[:, :-1])
    assert l_a == pytest.approx(l_b, rel=1e-14)
    np.testing.assert_allclose(d_a, d_b, rtol=0, atol=0)
    # a repeated index adds its probabilities
    idx3 = idx.copy(); idx3[:, 1] = idx3[:, 0]
    l_c, _ = oracle.sparse_soft_ce(z, idx3, prob)
    idx4 = idx[:, [0] + list(range(2, idx.shape[1]))]
    prob4 = prob[:, [0] + list(range(2, idx.shape[1]))].copy()
    prob4[:, 0] += prob[:, 1]
    l_d, _ = oracle.sparse_soft_ce(z, idx4, prob4)
    assert l_c == pytest.approx(l_d, rel=1e-13)
    # SUM reduction is N times MEAN_VALID without a mask
    ls, dzs = oracle.sparse_soft_ce(z, idx, prob, reduction=SUM)
    lm, dzm = oracle.sparse_soft_ce(z, idx, prob, reduction=MEAN_VALID)
    assert ls == pytest.approx(lm * z.shape[0], rel=1e-13)


def test_all_masked_gives_zero():
    z, idx, prob = _sparse_case(N=5)
    loss, dz = oracle.sparse_soft_ce(z, idx, prob, np.zeros(5, np.uint8))
    assert loss == 0.0 and np.all(dz == 0.0)
