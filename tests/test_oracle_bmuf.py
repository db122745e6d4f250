"""Pins of the oracle's BMUF-NBM global step (§VI-B, eqs. (2)-(6)): special
cases that reduce to plain model averaging and to taking the single local
model, a closed form of the block momentum over several blocks computed in
exact rational arithmetic, the all-reduced-sum form of the average, and the
hyper-parameter relation of eq. (6).  CPU only."""

from fractions import Fraction

import numpy as np
import pytest

import oracle


def _grid(rng, shape, scale_bits=20, span=4000):
    """fp32 values k * 2^-scale_bits: sums and differences are exact."""
    return (rng.integers(-span, span, shape) * 2.0 ** -scale_bits).astype(np.float32)


def test_single_worker_without_momentum_takes_the_local_model():
    # N = 1, eta = 0, zeta = 1: G = W - W_g, Delta = G, W_g(t) = W exactly
    rng = np.random.default_rng(0)
    n = 5000
    wg = (rng.standard_normal(n) * 0.05).astype(np.float32)
    w = (wg + rng.standard_normal(n).astype(np.float32) * 1e-3).astype(np.float32)
    d0 = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    new_w, d, bits = oracle.bmuf_block_update(w[None, :], 1, wg, d0, 0.0, 0.0, 1.0)
    np.testing.assert_array_equal(new_w.view(np.uint32), w.view(np.uint32))
    np.testing.assert_array_equal(bits, oracle.bf16_bits(w))
    np.testing.assert_array_equal(d, (w.astype(np.float64) - wg.astype(np.float64)).astype(np.float32))


@pytest.mark.parametrize("workers", [2, 4, 8])
def test_without_momentum_is_model_averaging(workers):
    # eta = 0, zeta = 1: W_g(t) is the plain average of eq. (2), here exact
    rng = np.random.default_rng(workers)
    n = 300
    models = _grid(rng, (workers, n))
    wg = _grid(rng, n)
    new_w, d, _ = oracle.bmuf_block_update(models, workers, wg, np.zeros(n, np.float32), 0.0, 0.0, 1.0)
    for j in range(n):
        mean = sum(Fraction(float(models[i, j])) for i in range(workers)) / workers
        assert Fraction(float(new_w[j])) == mean, j


def test_block_momentum_closed_form_over_blocks():
    # every worker ends each block at W_g(t-1) + c_i with mean(c_i) = c, so
    # G(t) = c every block and, from Delta(0) = 0 with constant eta and zeta,
    #   Delta(t) = zeta c (1 - eta^t) / (1 - eta),
    #   W_g(t)   = W_g(0) + (1 + eta) sum_{s<=t} Delta(s).
    rng = np.random.default_rng(7)
    n, N, blocks = 64, 4, 6
    eta, zeta = 0.5, 0.75
    c = _grid(rng, n, scale_bits=16, span=50)
    spread = _grid(rng, (N, n), scale_bits=16, span=20)
    spread -= spread.mean(axis=0, dtype=np.float64).astype(np.float32)  # exact: grid / 4
    wg = _grid(rng, n, scale_bits=12, span=1000)
    wg0 = wg.copy()
    d = np.zeros(n, np.float32)
    for t in range(1, blocks + 1):
        models = wg[None, :] + c[None, :] + spread
        wg, d, _ = oracle.bmuf_block_update(models, N, wg, d, eta, eta, zeta)
    E, Z = Fraction(eta), Fraction(zeta)
    for j in range(n):
        cj = Fraction(float(c[j]))
        deltas = [Z * cj * (1 - E ** s) / (1 - E) for s in range(1, blocks + 1)]
        ref_w = Fraction(float(wg0[j])) + (1 + E) * sum(deltas)
        assert abs(float(Fraction(float(d[j])) - deltas[-1])) <= 1e-6 * (abs(float(deltas[-1])) + 1e-12)
        assert abs(float(Fraction(float(wg[j])) - ref_w)) <= 1e-6 * (abs(float(ref_w)) + 1e-9)


def test_look_ahead_uses_the_next_momentum():
    # eta_t = 0 and eta_{t+1} = 0.9 from Delta(t-1) != 0: Delta(t) = zeta G and
    # W_g(t) = W_g(t-1) + (1 + eta_{t+1}) zeta G; the old Delta drops out
    rng = np.random.default_rng(3)
    n, N = 200, 2
    models = _grid(rng, (N, n))
    wg = _grid(rng, n)
    d0 = _grid(rng, n)
    new_w, d, _ = oracle.bmuf_block_update(models, N, wg, d0, 0.0, 0.9, 0.5)
    for j in range(n):
        G = (Fraction(float(models[0, j])) + Fraction(float(models[1, j]))) / 2 - Fraction(float(wg[j]))
        dj = Fraction(0.5) * G
        assert Fraction(float(d[j])) == dj
        ref = Fraction(float(wg[j])) + (1 + Fraction(np.float64(np.float32(0.9)))) * dj
        assert abs(float(Fraction(float(new_w[j])) - ref)) <= 2.0 ** -24 * abs(float(ref)) + 1e-30


def test_all_reduced_sum_gives_the_same_step():
    # the average may arrive as one pre-summed addend divided by N
    rng = np.random.default_rng(11)
    n, N = 1000, 8
    models = _grid(rng, (N, n))
    total = models.astype(np.float64).sum(axis=0).astype(np.float32)  # exact on the grid
    wg = _grid(rng, n)
    d0 = _grid(rng, n)
    a = oracle.bmuf_block_update(models, N, wg, d0, 0.875, 0.875, 1.5)
    b = oracle.bmuf_block_update(total[None, :], N, wg, d0, 0.875, 0.875, 1.5)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(np.asarray(x).view(np.uint32) if x.dtype == np.float32 else x,
                                      np.asarray(y).view(np.uint32) if y.dtype == np.float32 else y)


@pytest.mark.parametrize("C,N,eta", [(1.0, 8, 0.875), (2.0, 64, 0.9), (1.5, 1, 0.0)])
def test_eq5_hyper_parameters(C, N, eta):
    zeta = oracle.bmuf_zeta(C, N, eta)
    assert zeta / (N * (1.0 - eta)) == pytest.approx(C, rel=1e-15)
