"""Pins the oracle's column scores (squared per-column norms) against exact
rational arithmetic, closed-form special cases and the Frobenius identity."""
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import colnorm, k_from_ratio, select_topk, widen
from tests._golden import read_keyvals


def bf16_bits(rng, shape, emin, emax, zero_frac=0.0):
    """Random bf16 patterns: random sign, exponent in [emin, emax], 7-bit mantissa."""
    sign = rng.integers(0, 2, size=shape).astype(np.uint32) << 15
    exp = (rng.integers(emin, emax + 1, size=shape) + 127).astype(np.uint32) << 7
    man = rng.integers(0, 128, size=shape).astype(np.uint32)
    bits = (sign | exp | man).astype(np.uint16)
    if zero_frac:
        bits[rng.random(shape) < zero_frac] = 0
    return bits


def exact_colnorm(bits):
    """Column sums of squares as exact rationals."""
    n, m = bits.shape
    vals = widen(bits)
    return [sum((Fraction(float(vals[i, j])) ** 2 for i in range(n)), Fraction(0)) for j in range(m)]


@pytest.mark.parametrize("n,m,seed", [(1, 5, 0), (3, 7, 1), (17, 9, 2), (32, 33, 3), (5, 64, 4)])
def test_exactly_rounded_when_sum_fits_double(n, m, seed):
    # Exponents in [-6, 6]: squares carry 16 significant bits and span < 2^41,
    # so the exact sum of up to 32 of them fits a double; float(Fraction) is
    # then exact and one fp32 conversion is the correctly rounded result.
    rng = np.random.default_rng(seed)
    bits = bf16_bits(rng, (n, m), -6, 6, zero_frac=0.1)
    want = np.array([float(v) for v in exact_colnorm(bits)]).astype(np.float32)
    got = colnorm(bits)
    assert got.dtype == np.float32 and got.shape == (m,)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_within_one_ulp_of_exact_for_wide_exponents(seed):
    rng = np.random.default_rng(seed)
    bits = bf16_bits(rng, (40, 12), -60, 60)
    exact = exact_colnorm(bits)
    got = colnorm(bits)
    for j in range(12):
        err = abs(Fraction(float(got[j])) - exact[j])
        assert err <= exact[j] * Fraction(1, 1 << 23)


def test_single_row_is_square():
    rng = np.random.default_rng(5)
    bits = bf16_bits(rng, (1, 300), -60, 60)
    g = widen(bits[0]).astype(np.float64)
    assert np.array_equal(colnorm(bits), (g * g).astype(np.float32))


def test_zero_column_and_power_of_two_column():
    n, m = 37, 4
    bits = np.zeros((n, m), dtype=np.uint16)
    e = -5
    two_e = np.array([2.0 ** e], dtype=np.float32).view(np.uint32)[0] >> 16
    bits[:, 1] = two_e
    bits[::2, 1] |= 0x8000  # alternate signs
    bits[:, 3] = 0x8000     # -0.0 everywhere
    s = colnorm(bits)
    assert s[0] == 0 and s[3] == 0
    assert s[1] == np.float32(n * 2.0 ** (2 * e))


def test_transpose_is_caught():
    bits = np.zeros((3, 5), dtype=np.uint16)
    bits[2, 4] = 0x4040  # 3.0
    s = colnorm(bits)
    assert s.tolist() == [0, 0, 0, 0, 9.0]


def test_empty_rows_give_zero_scores():
    assert np.array_equal(colnorm(np.zeros((0, 6), np.uint16)), np.zeros(6, np.float32))


@pytest.mark.parametrize("seed", [11, 12])
def test_frobenius_identity_split_by_selection(seed):
    rng = np.random.default_rng(seed)
    bits = bf16_bits(rng, (64, 200), -20, 20)
    s = colnorm(bits)
    frob = math.fsum(float(v) * float(v) for v in widen(bits).ravel())
    sel = select_topk(s, k_from_ratio(0.1, 200))
    part = math.fsum(float(x) for x in s[sel.sel]) + math.fsum(float(x) for x in s[sel.unsel])
    assert abs(part - frob) <= 1e-7 * frob


def test_score_vector_size_matches_paper():
    g = read_keyvals("paper_numbers.txt")
    n, m = g["qproj_rows"], g["qproj_cols"]
    bits = np.full((n, m), 0x3F80, dtype=np.uint16)  # 1.0
    s = colnorm(bits)
    assert s.size == g["score_vector_entries"] and s.nbytes == g["score_vector_bytes"]
    assert (s == np.float32(n)).all()
