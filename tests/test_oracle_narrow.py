"""Narrower-mantissa inputs (App. "PAM with Narrower Mantissas", reading R11):
the oracle's rounding against library conversions, exact rationals and
invariants, its two forms against each other, planted mistakes, and the narrow
matrix product's special cases."""
import numpy as np
import pytest

from narrow_pins import CHECKS, INF, SIGN, bits, sample
from oracle import pam_ref


@pytest.mark.parametrize("check", CHECKS, ids=lambda c: c.__name__)
def test_rounding_pins(check):
    check(pam_ref.round_mantissa_ref)


def test_vector_form_equals_scalar_form():
    x = sample(100000, 5)
    for b in range(0, 24):
        assert np.array_equal(bits(pam_ref.round_mantissa_ref(x, b)), bits(pam_ref.round_mantissa_scalar_ref(x, b))), b


def mutant(kind):
    def rnd(x, b):
        x = np.asarray(x, np.float32)
        u = x.view(np.uint32).astype(np.int64)
        if b == 23:
            return x.copy()
        drop = 23 - b
        low, kept, half = u & ((1 << drop) - 1), u >> drop, 1 << (drop - 1)
        if kind == "truncate":
            up = np.zeros_like(low, dtype=bool)
        elif kind == "ties_away":
            up = low >= half
        elif kind == "ties_down":
            up = low > half
        else:
            up = (low > half) | ((low == half) & ((kept & 1) == 1))
        r = (kept + up) << drop
        if kind == "no_carry":
            r = (u & ~np.int64(0x7FFFFF)) | (r & 0x7FFFFF)
        if kind == "saturate":
            r = np.where(((r & INF) == INF) & ((u & INF) != INF), (r & SIGN) | 0x7F7FFFFF & ~((1 << drop) - 1), r)
        if kind != "rounds_nan":
            r = np.where((u & INF) == INF, u, r)
        return r.astype(np.uint32).view(np.float32)
    return rnd


@pytest.mark.parametrize("kind", ["truncate", "ties_away", "ties_down", "no_carry", "saturate"])
def test_rounding_mutants_are_caught(kind):
    caught = False
    for check in CHECKS:
        try:
            check(mutant(kind))
        except AssertionError:
            caught = True
            break
    assert caught, kind


def test_narrow_product_special_cases():
    """Inputs already on the m-bit grid: the narrow product is the plain PAM
    product; and rounding commutes with transposition."""
    g = np.random.default_rng(6)
    a = pam_ref.round_mantissa_ref(g.standard_normal((9, 13)).astype(np.float32), 4)
    b = pam_ref.round_mantissa_ref(g.standard_normal((13, 7)).astype(np.float32), 4)
    c0, _ = pam_ref.pam_gemm_ref(a, b)
    c1, _ = pam_ref.pam_gemm_ref(pam_ref.round_mantissa_ref(a, 4), pam_ref.round_mantissa_ref(b, 4))
    assert np.array_equal(c0, c1)
    assert np.array_equal(pam_ref.round_mantissa_ref(a.T, 3), pam_ref.round_mantissa_ref(a, 3).T)
