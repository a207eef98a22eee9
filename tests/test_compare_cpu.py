"""The comparator's exact fp32 helpers (tests/compare.py), pinned on the CPU: the order key is
monotone in the value, and the fused multiply-add check accepts exactly the correctly rounded
result (ties to even) and rejects a neighbour."""
from fractions import Fraction

import numpy as np
import pytest

from tests import compare


def test_order_key_is_monotone():
    x = np.array([-np.inf, -3.5, -1e-30, -0.0, 0.0, 1e-38, 2.0, np.inf], dtype=np.float32)
    k = compare.order_key(x)
    assert np.all(np.diff(k.astype(np.int64)) > 0)
    rng = np.random.default_rng(5)
    y = (rng.standard_normal(10000) * 10.0 ** rng.integers(-20, 20, 10000)).astype(np.float32)
    order = np.argsort(y, kind="stable")
    assert np.all(np.diff(compare.order_key(y[order]).astype(np.int64)) >= 0)


def _fma_exact(a, b, c):
    return compare._round_f32_exact(Fraction(float(np.float32(a))) * Fraction(float(np.float32(b)))
                                    + Fraction(float(np.float32(c))))


def test_exact_rounding_ties_to_even():
    # 1 + 2^-24 lies halfway between 1 and 1 + 2^-23: the even significand (1) wins;
    # 1 + 3 * 2^-24 lies halfway between 1 + 2^-23 and 1 + 2^-22: 1 + 2^-22 (even) wins
    one = np.float32(1.0)
    assert compare._round_f32_exact(Fraction(1) + Fraction(1, 2 ** 24)) == one
    assert compare._round_f32_exact(Fraction(1) + Fraction(3, 2 ** 24)) == np.float32(1 + 2 ** -22)
    assert compare._round_f32_exact(Fraction(1) + Fraction(3, 2 ** 25)) == np.float32(1 + 2 ** -23)


@pytest.mark.parametrize("seed", [0, 1])
def test_fma_check_accepts_the_fused_result_and_rejects_a_neighbour(seed):
    rng = np.random.default_rng(seed)
    a = np.float32(rng.uniform(0.1, 3.0))
    b = (rng.standard_normal(300) * 1e-3).astype(np.float32)
    c = (rng.standard_normal(300) * 1e-3).astype(np.float32)
    want = np.array([_fma_exact(a, x, y) for x, y in zip(b, c)], dtype=np.float32)
    compare.assert_fma_f32(want, float(a), b, c, "fma")
    for i in (0, 7, 299):
        bad = want.copy()
        bad[i] = np.nextafter(bad[i], np.float32(np.inf))
        with pytest.raises(AssertionError):
            compare.assert_fma_f32(bad, float(a), b, c, "fma")


def test_fma_check_sees_a_separately_rounded_product():
    # a * b rounded to fp32 before the add differs from the fused result for these operands
    a, b, c = np.float32(1 + 2 ** -12), np.float32(1 + 2 ** -12), np.float32(-1.0)
    fused = _fma_exact(a, b, c)
    unfused = np.float32(np.float32(a * b) + c)
    assert fused != unfused
    compare.assert_fma_f32(np.array([fused]), float(a), np.array([b]), np.array([c]), "fma")
    with pytest.raises(AssertionError):
        compare.assert_fma_f32(np.array([unfused]), float(a), np.array([b]), np.array([c]), "fma")
