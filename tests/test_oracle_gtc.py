"""Pins of the oracle's gradient threshold compression: conservation (what is
sent plus what is kept equals what came in), a sequential brute-force
definition on small inputs, closed-form multi-step behaviour, adversarial
values, and the decode round trip.  CPU only."""

import os
import struct

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _sequential(grad, residual, tau):
    """Element-by-element definition with Python-level fp32 scalars."""
    f32 = np.float32
    tau = f32(tau)
    r_out, words = [], []
    for i, (g, r) in enumerate(zip(grad.tolist(), residual.tolist())):
        a = f32(f32(r) + f32(g))
        if a > tau:
            r_out.append(f32(a - tau)); words.append((i << 1) | 0)
        elif a < -tau:
            r_out.append(f32(a + tau)); words.append((i << 1) | 1)
        else:
            r_out.append(a)
    return np.array(r_out, np.float32), np.array(words, np.uint32)


def _bits(x):
    return np.asarray(x, np.float32).view(np.uint32)


def test_matches_sequential_definition():
    rng = np.random.default_rng(0)
    n, tau = 3000, 1e-3
    g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    r = (rng.standard_normal(n) * 5e-4).astype(np.float32)
    r[::97] = 0.0
    new_r, words, count = oracle.grad_threshold_encode(g, r, tau)
    sr, sw = _sequential(g, r, tau)
    np.testing.assert_array_equal(_bits(new_r), _bits(sr))
    np.testing.assert_array_equal(words, sw)
    assert count == sw.shape[0]


def test_conservation_exact_on_power_of_two_grid():
    # values k * 2^-20 with tau = 2^-10: every add and subtract is exact, so
    # sent + kept must equal residual + gradient exactly.
    rng = np.random.default_rng(1)
    n = 200_000
    tau = np.float32(2.0 ** -10)
    g = (rng.integers(-5000, 5000, n) * 2.0 ** -20).astype(np.float32)
    r = (rng.integers(-1500, 1500, n) * 2.0 ** -20).astype(np.float32)
    new_r, words, count = oracle.grad_threshold_encode(g, r, tau)
    sent = oracle.grad_threshold_decode(words, count, tau, n)
    lhs = new_r.astype(np.float64) + sent.astype(np.float64)
    rhs = r.astype(np.float64) + g.astype(np.float64)
    np.testing.assert_array_equal(lhs, rhs)
    assert np.all(np.abs(new_r) <= np.abs(r.astype(np.float64) + g) )
    assert 0 < count < n


def test_conservation_within_rounding_for_random_fp32():
    rng = np.random.default_rng(2)
    n, tau = 100_000, np.float32(1e-4)
    g = (rng.standard_normal(n) * 3e-4).astype(np.float32)
    r = (rng.standard_normal(n) * 1e-4).astype(np.float32)
    new_r, words, count = oracle.grad_threshold_encode(g, r, tau)
    sent = oracle.grad_threshold_decode(words, count, tau, n)
    exact = r.astype(np.float64) + g.astype(np.float64)
    a = (r + g).astype(np.float64)
    err = new_r.astype(np.float64) + sent.astype(np.float64) - exact
    bound = 0.5 * np.spacing(np.abs(a).astype(np.float32)).astype(np.float64) \
        + 0.5 * np.spacing(np.abs(new_r)).astype(np.float64)
    assert np.all(np.abs(err) <= bound)


def test_closed_form_drain_from_golden():
    # tests/golden/gtc_drain.txt: tau = 2^-10, r0 = 5.5 tau, zero gradients.
    spec = {}
    with open(os.path.join(GOLDEN, "gtc_drain.txt")) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if line:
                k, v = line.split("=")
                spec[k.strip()] = v.strip()
    tau = np.float32(float.fromhex(spec["tau"]))
    r = np.full(4, np.float32(float.fromhex(spec["r0"])), np.float32)
    r[1] = -r[1]
    g = np.zeros(4, np.float32)
    words_per_call = [int(w) for w in spec["words_per_call"].split(",")]
    for call, expected in enumerate(words_per_call):
        r, words, count = oracle.grad_threshold_encode(g, r, tau)
        assert count == expected, call
        if count:
            np.testing.assert_array_equal(words, [(i << 1) | (i == 1) for i in range(4)])
    assert r[0] == np.float32(float.fromhex(spec["r_final"]))
    assert r[1] == -np.float32(float.fromhex(spec["r_final"]))


def test_huge_tau_sends_nothing_and_accumulates():
    rng = np.random.default_rng(3)
    g = rng.standard_normal(1000).astype(np.float32)
    r = rng.standard_normal(1000).astype(np.float32)
    new_r, words, count = oracle.grad_threshold_encode(g, r, np.float32(np.inf))
    assert count == 0 and words.shape == (0,)
    np.testing.assert_array_equal(_bits(new_r), _bits(r + g))


def test_adversarial_values():
    tau = np.float32(0.5)
    f = np.float32
    sub = np.array([1], np.uint32).view(np.float32)[0]           # smallest subnormal
    r = np.array([0, 0, 0, 0, 0, 0, -0.0, sub, 0, 0, 0, 0, 1e30], np.float32)
    g = np.array([0.5, -0.5, np.nextafter(f(0.5), f(1)), -np.nextafter(f(0.5), f(1)),
                  1.0, -1.75, -0.0, sub, np.inf, -np.inf, np.nan, 3e38, 3e38], np.float32)
    new_r, words, count = oracle.grad_threshold_encode(g, r, tau)
    sr, sw = _sequential(g, r, tau)
    np.testing.assert_array_equal(_bits(new_r), _bits(sr))
    np.testing.assert_array_equal(words, sw)
    expected_words = [(2 << 1), (3 << 1) | 1, (4 << 1), (5 << 1) | 1, (8 << 1), (9 << 1) | 1,
                      (11 << 1), (12 << 1)]
    np.testing.assert_array_equal(words, expected_words)
    assert new_r[0] == f(0.5) and new_r[1] == f(-0.5)          # exactly tau: kept
    assert new_r[4] == f(0.5) and new_r[5] == f(-1.25)         # one quantum only
    assert _bits(new_r[6]) == _bits(f(-0.0))                   # -0 + -0 = -0
    assert _bits(new_r[7]) == 2                                # subnormals kept exact
    assert np.isposinf(new_r[8]) and np.isneginf(new_r[9])
    assert np.isnan(new_r[10])                                 # NaN never sent


def test_decode_modes_and_word_format():
    rng = np.random.default_rng(4)
    n, tau = 5000, np.float32(2e-3)
    g = (rng.standard_normal(n) * 3e-3).astype(np.float32)
    r = np.zeros(n, np.float32)
    new_r, words, count = oracle.grad_threshold_encode(g, r, tau)
    assert np.all(np.diff(words >> 1) > 0)                     # strictly ascending
    dense = oracle.grad_threshold_decode(words, count, tau, n)
    idx = words >> 1
    assert np.all(dense[idx] == np.where(words & 1, -tau, tau))
    mask = np.ones(n, bool); mask[idx] = False
    assert np.all(_bits(dense[mask]) == 0)                     # +0.0 elsewhere
    base = rng.standard_normal(n).astype(np.float32)
    acc = oracle.grad_threshold_decode(words, count, tau, n, dense=base, accumulate=True)
    np.testing.assert_array_equal(_bits(acc), _bits(base + dense))
    # the word packs a 31-bit index and the sign in bit 0
    w = struct.unpack("<I", struct.pack("<I", (12345 << 1) | 1))[0]
    assert (w >> 1, w & 1) == (12345, 1)


# ---- aggregate of several workers' sparse updates ---------------------------

def _streams(rng, S, n, tau, scale=1.5e-3):
    """S workers' encodes of their own gradients; [S][n] words, counts."""
    words = np.zeros((S, n), np.uint32)
    counts = np.zeros(S, np.int64)
    rs, gs = [], []
    for s in range(S):
        g = (rng.integers(-6000, 6000, n) * 2.0 ** -22).astype(np.float32)
        r = (rng.integers(-1000, 1000, n) * 2.0 ** -22).astype(np.float32)
        new_r, w, c = oracle.grad_threshold_encode(g, r, tau)
        words[s, :c] = w
        words[s, c:] = 0xFFFFFFFF  # garbage past the count
        counts[s] = c
        rs.append((r, g, new_r))
    return words, counts, rs


@pytest.mark.parametrize("accumulate", [False, True])
def test_decode_multi_single_stream_is_decode(accumulate):
    rng = np.random.default_rng(20)
    n, tau = 20_000, np.float32(1e-3)
    g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    _, w, c = oracle.grad_threshold_encode(g, np.zeros(n, np.float32), tau)
    base = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    a = oracle.grad_threshold_decode(w, c, tau, n, base, accumulate)
    b = oracle.grad_threshold_decode_multi(w[None, :], [c], tau, n, base, accumulate)
    np.testing.assert_array_equal(_bits(a), _bits(b))


def test_decode_multi_equals_sum_of_single_decodes():
    # tau a power of two: each single decode is exact, their fp64 sum too
    rng = np.random.default_rng(21)
    n, S, tau = 30_000, 6, np.float32(2.0 ** -10)
    words, counts, _ = _streams(rng, S, n, tau)
    total = np.zeros(n, np.float64)
    for s in range(S):
        total += oracle.grad_threshold_decode(words[s], counts[s], tau, n).astype(np.float64)
    agg = oracle.grad_threshold_decode_multi(words, counts, tau, n)
    np.testing.assert_array_equal(agg.astype(np.float64), total)
    assert np.count_nonzero(np.abs(total) > tau) > 0  # some indices sent by several workers


def test_decode_multi_is_order_independent():
    rng = np.random.default_rng(22)
    n, S, tau = 10_000, 5, np.float32(1e-3)
    words, counts, _ = _streams(rng, S, n, tau)
    base = (rng.standard_normal(n) * 1e-2).astype(np.float32)
    a = oracle.grad_threshold_decode_multi(words, counts, tau, n, base, True)
    perm = rng.permutation(S)
    b = oracle.grad_threshold_decode_multi(words[perm], counts[perm], tau, n, base, True)
    np.testing.assert_array_equal(_bits(a), _bits(b))


def test_decode_multi_conserves_across_workers():
    # sum over workers of (kept + sent) equals sum of (residual + gradient),
    # exactly on the power-of-two grid
    rng = np.random.default_rng(23)
    n, S, tau = 25_000, 4, np.float32(2.0 ** -10)
    words, counts, rs = _streams(rng, S, n, tau)
    agg = oracle.grad_threshold_decode_multi(words, counts, tau, n).astype(np.float64)
    kept = sum(x[2].astype(np.float64) for x in rs)
    came = sum(x[0].astype(np.float64) + x[1].astype(np.float64) for x in rs)
    np.testing.assert_array_equal(kept + agg, came)


def test_decode_multi_cancelling_signs():
    n, tau = 8, np.float32(0.25)
    words = np.array([[(3 << 1) | 0, (5 << 1) | 0], [(3 << 1) | 1, (5 << 1) | 0]], np.uint32)
    out = oracle.grad_threshold_decode_multi(words, [2, 2], tau, n)
    np.testing.assert_array_equal(out, np.array([0, 0, 0, 0, 0, 0.5, 0, 0], np.float32))
    assert not np.signbit(out[3])
    base = np.full(n, 1.0, np.float32)
    acc = oracle.grad_threshold_decode_multi(words, [2, 2], tau, n, base, True)
    np.testing.assert_array_equal(acc, np.array([1, 1, 1, 1, 1, 1.5, 1, 1], np.float32))
    # accumulate leaves elements no word names untouched, -0.0 included
    negz = np.full(n, -0.0, np.float32)
    acc = oracle.grad_threshold_decode_multi(words, [2, 2], tau, n, negz, True)
    assert np.all(np.signbit(acc[[0, 1, 2, 4, 6, 7]]))
    assert not np.signbit(acc[3]) and acc[5] == 0.5
