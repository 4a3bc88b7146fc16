"""Pins of the oracle's history quantiser (Sec. 3, Table 1) to facts outside it.

Decimal rounding is checked against Python's `decimal` module (a library
implementation of k-significant-digit rounding with ties away from zero),
against a brute-force nearest-grid-point search, against hand-worked values,
and against the properties the method relies on (idempotence, monotonicity,
code equality <=> value equality).
"""
import decimal
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import Q_EXACT, Q_SIGDIG, Q_SIGN, code_words, dequantize, quantize
from oracle.rnnlm_oracle import dequantize_exact

TINY = Fraction(1, 10 ** 20)


def decimal_reference(x, k):
    """k significant digits, ROUND_HALF_UP = ties away from zero in `decimal`."""
    if abs(Fraction(float(x))) < TINY:
        return Fraction(0)
    ctx = decimal.Context(prec=k, rounding=decimal.ROUND_HALF_UP)
    return Fraction(ctx.plus(decimal.Decimal(float(x))))


def random_unit_floats(rng, n):
    # log-uniform magnitudes over [1e-22, 1] plus uniform ones, random signs
    mag = np.concatenate([10.0 ** rng.uniform(-22, 0, n // 2), rng.uniform(0, 1, n - n // 2)])
    x = (mag * rng.choice([-1.0, 1.0], n)).astype(np.float32)
    return np.clip(x, -1, 1).astype(np.float32)


@pytest.mark.parametrize("k", [1, 2, 3])
def test_sigdig_matches_decimal_module(k):
    rng = np.random.default_rng(1000 + k)
    x = random_unit_floats(rng, 20000)
    codes = quantize(x, Q_SIGDIG, k)
    for xi, ci in zip(x, codes):
        assert dequantize_exact(ci, Q_SIGDIG, k) == decimal_reference(xi, k), (xi, k)


def dyadic_ties(k):
    """fp32 values that lie exactly halfway between two k-digit decimals."""
    out = []
    for e in range(-6, 1):
        step = Fraction(10) ** (e - k + 1)
        for m in range(10 ** (k - 1), 10 ** k):
            mid = (m + Fraction(1, 2)) * step
            f = np.float32(float(mid))
            if Fraction(float(f)) == mid and abs(mid) <= 1:
                out.append(f)
    return np.array(out, np.float32)


@pytest.mark.parametrize("k", [1, 2, 3])
def test_sigdig_ties_round_away_from_zero(k):
    ties = dyadic_ties(k)
    assert len(ties) > 0
    for sgn in (1, -1):
        x = (sgn * ties).astype(np.float32)
        codes = quantize(x, Q_SIGDIG, k)
        for xi, ci in zip(x, codes):
            v = dequantize_exact(ci, Q_SIGDIG, k)
            assert abs(v) > abs(Fraction(float(xi)))     # away from zero
            assert v == decimal_reference(xi, k)


def test_sigdig_hand_worked_values():
    # 0.125 is a tie at 2 digits -> 0.13; 0.0625 -> 0.063 (k=2), exact at k=3
    cases = [(0.125, 2, Fraction(13, 100)), (0.0625, 2, Fraction(63, 1000)),
             (0.0625, 3, Fraction(625, 10000)), (1.0, 3, Fraction(1)),
             (-0.5, 1, Fraction(-1, 2)), (0.9996, 3, Fraction(1)),
             (0.95, 1, Fraction(9, 10)),     # fp32(0.95) is just below 0.95
             (0.01, 2, Fraction(1, 100)),    # fp32(0.01) < 0.01: rounds up into the next decade
             (-0.0, 2, Fraction(0)), (1e-21, 3, Fraction(0))]
    for x, k, want in cases:
        c = quantize(np.array([x], np.float32), Q_SIGDIG, k)[0]
        assert dequantize_exact(c, Q_SIGDIG, k) == want, (x, k)


def test_sigdig_brute_force_nearest_grid_point():
    """The code is the nearest k-digit decimal (ties: larger magnitude)."""
    rng = np.random.default_rng(7)
    for k, n in ((1, 60), (2, 60), (3, 20)):
        x = random_unit_floats(rng, n)
        x = x[np.abs(x) >= 1e-19]
        codes = quantize(x, Q_SIGDIG, k)
        for xi, ci in zip(x, codes):
            ax = abs(Fraction(float(xi)))
            best = None
            for e in range(-20, 1):
                for m in range(10 ** (k - 1), 10 ** k + 1):
                    c = m * Fraction(10) ** (e - k + 1)
                    d = abs(c - ax)
                    if best is None or d < best[0] or (d == best[0] and c > best[1]):
                        best = (d, c)
            want = best[1] if xi >= 0 else -best[1]
            assert dequantize_exact(ci, Q_SIGDIG, k) == want


@settings(max_examples=300, deadline=None)
@given(st.floats(min_value=-1.0, max_value=1.0, width=32), st.integers(1, 3))
def test_sigdig_idempotent(x, k):
    c1 = quantize(np.array([x], np.float32), Q_SIGDIG, k)
    y = dequantize(c1, Q_SIGDIG, k)
    c2 = quantize(y, Q_SIGDIG, k)
    assert c1[0] == c2[0]


@settings(max_examples=300, deadline=None)
@given(st.floats(min_value=-1.0, max_value=1.0, width=32),
       st.floats(min_value=-1.0, max_value=1.0, width=32), st.integers(1, 3))
def test_sigdig_monotone_and_code_equality(x, y, k):
    cx, cy = quantize(np.array([x, y], np.float32), Q_SIGDIG, k)
    vx, vy = dequantize_exact(cx, Q_SIGDIG, k), dequantize_exact(cy, Q_SIGDIG, k)
    if np.float32(x) <= np.float32(y):
        assert vx <= vy
    assert (cx == cy) == (vx == vy)


@settings(max_examples=300, deadline=None)
@given(st.floats(min_value=float(np.float32(1e-19)), max_value=1.0, width=32), st.integers(1, 3))
def test_sigdig_error_bound_and_symmetry(x, k):
    cp, cn = quantize(np.array([x, -x], np.float32), Q_SIGDIG, k)
    v = dequantize_exact(cp, Q_SIGDIG, k)
    assert dequantize_exact(cn, Q_SIGDIG, k) == -v
    ax = Fraction(float(np.float32(x)))
    e = 0
    while Fraction(10) ** e > ax:
        e -= 1
    assert abs(v - ax) <= Fraction(1, 2) * Fraction(10) ** (e - k + 1)


def test_sigdig_rejects_out_of_domain():
    for bad in (1.0000001, -1.5, np.inf, np.nan):
        with pytest.raises(ValueError):
            quantize(np.array([0.5, bad], np.float32), Q_SIGDIG, 2)


def test_sign_quantiser():
    x = np.array([0.3, -0.3, 0.0, -0.0, 1.0, -1e-30], np.float32)
    c = quantize(x, Q_SIGN)
    d = dequantize(c, Q_SIGN)
    assert set(np.unique(d)) <= {-1.0, 1.0}
    assert list(d) == [1, -1, 1, 1, 1, -1]
    assert np.array_equal(quantize(d, Q_SIGN), c)          # idempotent


def test_exact_quantiser_identifies_signed_zeros():
    x = np.array([0.0, -0.0, 0.25, -0.25], np.float32)
    c = quantize(x, Q_EXACT)
    assert c[0] == c[1] and c[2] != c[3]
    assert np.array_equal(dequantize(c, Q_EXACT), np.array([0, 0, 0.25, -0.25], np.float32))


def test_code_word_packing_matches_numpy_packbits():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, 256)).astype(np.float32)
    bits = quantize(x, Q_SIGN)
    w = code_words(bits, Q_SIGN)
    ref = np.packbits(bits, axis=1, bitorder="little").view("<u8")
    assert np.array_equal(w, ref)
    c16 = quantize(np.tanh(x), Q_SIGDIG, 2)
    assert np.array_equal(code_words(c16, Q_SIGDIG), c16.astype("<u2").view("<u8"))
    c32 = quantize(x, Q_EXACT)
    assert np.array_equal(code_words(c32, Q_EXACT), c32.astype("<u4").view("<u8"))
