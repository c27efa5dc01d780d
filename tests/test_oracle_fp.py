"""Pins of the oracle's rounding helpers (CPU only): IEEE semantics checked
against numpy / PyTorch casts and against brute-force nearest-value search."""
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import fp as OF


def _specials():
    f = np.float32
    vals = [0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, np.finfo(f).max, -np.finfo(f).max,
            np.finfo(f).tiny, 1e-45, -1e-45, 65504.0, 65520.0, 6e-8, 3.0e-5]
    # bf16 halfway cases: 1 + 2^-8 (tie -> even 1.0), 1 + 3*2^-8 (tie -> up)
    vals += [1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -8 + 2.0 ** -20]
    # fp16 halfway cases
    vals += [1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11, 2049.0, 2051.0]
    return np.array(vals, dtype=np.float32)


def test_bf16_matches_torch():
    rng = np.random.Generator(np.random.PCG64(0))
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 20000),
                        _specials()]).astype(np.float32)
    ours = OF.round_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))


def test_bf16_nan_kept():
    x = np.array([np.nan, -np.nan], dtype=np.float32)
    assert np.all(np.isnan(OF.round_bf16(x)))


def test_f16_matches_torch():
    rng = np.random.Generator(np.random.PCG64(1))
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32) * 2.0 ** rng.integers(-26, 18, 20000),
                        _specials()]).astype(np.float32)
    ours = OF.round_f16(x)
    ref = torch.from_numpy(x).to(torch.float16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))


def _f32_neighbours(v):
    v = np.float32(v)
    return [np.nextafter(v, np.float32(-np.inf)), v, np.nextafter(v, np.float32(np.inf))]


def test_fraction_to_f32_is_nearest():
    import random
    rnd = random.Random(7)
    cases = [Fraction(1, 3), Fraction(-8, 3), Fraction(1, 6), Fraction(4, 3), Fraction(1, 24),
             Fraction(-1, 12), Fraction(2 ** 30 + 1, 2 ** 30), Fraction(1, 10 ** 40)]
    cases += [Fraction(rnd.randint(-10 ** 9, 10 ** 9), rnd.randint(1, 10 ** 9)) for _ in range(300)]
    for q in cases:
        r = OF.fraction_to_f32(q)
        rf = Fraction(r)
        assert np.float32(r) == r            # representable in fp32
        for nb in _f32_neighbours(r):
            if np.isfinite(nb):
                assert abs(Fraction(float(nb)) - q) >= abs(rf - q)


def test_fraction_to_f32_ties_to_even():
    one = Fraction(1)
    ulp = Fraction(1, 2 ** 23)
    assert OF.fraction_to_f32(one + ulp / 2) == 1.0                  # tie, even is 1.0
    assert OF.fraction_to_f32(one + 3 * ulp / 2) == float(one + 2 * ulp)  # tie, even is up
    assert OF.fraction_to_f32(Fraction(3, 2 ** 150)) == float(Fraction(2, 2 ** 149))  # subnormal
    assert OF.fraction_to_f32(Fraction(2 ** 129)) == float("inf")


@pytest.mark.parametrize("q", [Fraction(1, 2), Fraction(-5, 4), Fraction(3), Fraction(0)])
def test_fraction_to_f32_exact_values(q):
    assert OF.fraction_to_f32(q) == float(q)


def test_fma_f32_is_correctly_rounded():
    """fma_f32 against the exact rational a*b + c rounded once by
    fraction_to_f32 (itself pinned by brute force above), on random triples of
    spread exponents, on cancelling triples (c close to -a*b), and on a triple
    whose float64 sum lands exactly half-way between two fp32 numbers while
    the exact sum does not (a naive double rounding picks the wrong side)."""
    rng = np.random.default_rng(11)
    n = 4000
    a = (rng.standard_normal(n) * 2.0 ** rng.integers(-20, 20, n)).astype(np.float32)
    b = (rng.standard_normal(n) * 2.0 ** rng.integers(-20, 20, n)).astype(np.float32)
    c = (rng.standard_normal(n) * 2.0 ** rng.integers(-40, 40, n)).astype(np.float32)
    cancel = rng.random(n) < 0.3
    c[cancel] = (-(a[cancel].astype(np.float64) * b[cancel].astype(np.float64))).astype(np.float32)
    got = OF.fma_f32(a, b, c)
    for i in range(n):
        exact = Fraction(float(a[i])) * Fraction(float(b[i])) + Fraction(float(c[i]))
        assert float(got[i]) == OF.fraction_to_f32(exact), i
    # p = 2^-24 (1 + 2^-23)(1 - 2^-23) = 2^-24 - 2^-70 and c = 1 + 2^-23: the
    # float64 sum is the midpoint 1 + 2^-23 + 2^-24; the exact sum is just below
    a1 = np.float32(2.0 ** -24 * (1 + 2.0 ** -23))
    b1 = np.float32(1 - 2.0 ** -23)
    c1 = np.float32(1 + 2.0 ** -23)
    naive = np.float32(np.float64(a1) * np.float64(b1) + np.float64(c1))
    assert float(naive) == 1 + 2.0 ** -22
    assert float(OF.fma_f32(a1, b1, c1)) == 1 + 2.0 ** -23
