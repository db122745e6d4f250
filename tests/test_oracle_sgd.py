"""Pins of the oracle's bf16 rounding (against torch's fp32 -> bf16 cast, a
library routine) and of the SGD step (closed forms, exact rational
arithmetic).  CPU only."""

from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle


def _torch_bf16_bits(x32):
    t = torch.from_numpy(np.ascontiguousarray(x32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_bf16_rounding_matches_torch_on_every_exponent_and_tie_class():
    hi = np.arange(1 << 16, dtype=np.uint32) << np.uint32(16)
    lows = np.array([0x0000, 0x0001, 0x3FFF, 0x7FFF, 0x8000, 0x8001, 0xBFFF, 0xFFFF],
                    dtype=np.uint32)
    bits = (hi[:, None] | lows[None, :]).ravel()
    x = bits.view(np.float32)
    ours = oracle.bf16_bits(x)
    ref = _torch_bf16_bits(x)
    nan = np.isnan(x)
    np.testing.assert_array_equal(ours[~nan], ref[~nan])
    # NaN: both give a quiet NaN
    assert np.all(np.isnan(oracle.bf16_bits_to_f32(ours[nan])))
    assert np.all(np.isnan(oracle.bf16_bits_to_f32(ref[nan])))


def test_bf16_rounding_matches_torch_on_random_patterns():
    bits = np.random.default_rng(0).integers(0, 1 << 32, size=1 << 22, dtype=np.uint64)
    x = bits.astype(np.uint32).view(np.float32)
    ours = oracle.bf16_bits(x)
    ref = _torch_bf16_bits(x)
    ok = ~np.isnan(x)
    np.testing.assert_array_equal(ours[ok], ref[ok])


def test_sgd_closed_forms():
    rng = np.random.default_rng(1)
    w = rng.standard_normal(1000).astype(np.float32)
    u = rng.standard_normal(1000).astype(np.float32)
    new, _ = oracle.sgd_apply(w, u, 0.0)
    np.testing.assert_array_equal(new, w)
    new, _ = oracle.sgd_apply(w, np.zeros_like(u), 0.37)
    np.testing.assert_array_equal(new, w)
    # powers of two: exact
    w2 = np.array([1.0, -2.0, 0.75], np.float32)
    u2 = np.array([0.5, 0.25, -1.0], np.float32)
    new, bits = oracle.sgd_apply(w2, u2, 0.5)
    np.testing.assert_array_equal(new, np.array([0.75, -2.125, 1.25], np.float32))
    np.testing.assert_array_equal(bits, oracle.bf16_bits(new))


def test_sgd_is_correctly_rounded_almost_always():
    # fp64 evaluation then one rounding to fp32 equals the correctly rounded
    # exact result except on rare double-rounding ties, and is never more than
    # one ulp away.
    rng = np.random.default_rng(2)
    n = 4000
    w = rng.standard_normal(n).astype(np.float32)
    u = (rng.standard_normal(n) * 10).astype(np.float32)
    lr = np.float32(0.01)
    new, _ = oracle.sgd_apply(w, u, lr)
    mismatches = 0
    for i in range(n):
        exact = Fraction(float(w[i])) - Fraction(float(lr)) * Fraction(float(u[i]))
        lo = np.float32(float(exact))   # float() is correctly rounded to fp64
        # correctly rounded fp32 of the exact rational
        cands = [np.nextafter(lo, np.float32(-np.inf)), lo, np.nextafter(lo, np.float32(np.inf))]
        best = min(cands, key=lambda c: (abs(Fraction(float(c)) - exact),
                                         int(np.asarray(c).view(np.uint32)) & 1))
        if best != new[i]:
            mismatches += 1
            assert abs(Fraction(float(new[i])) - exact) <= Fraction(float(np.spacing(best)))
    assert mismatches <= n // 1000
