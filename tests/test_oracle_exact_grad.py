"""The exact derivative of PAM products (Table 1, reading R15), pinned by
finite differences of the PAM oracle itself, by true multiplication where one
operand is a power of two, and by its zero cases."""
import numpy as np
import pytest

from oracle import pam_ref


def next_away(x):
    """The float32 one ulp further from zero."""
    x = np.asarray(x, np.float32)
    return np.nextafter(x, np.where(x < 0, np.float32(-np.inf), np.float32(np.inf)).astype(np.float32))


def normal_values(shape, seed, lo=-20, hi=20):
    g = np.random.default_rng(seed)
    e = g.integers(lo, hi, size=shape)
    m = g.integers(0, 1 << 23, size=shape)
    s = g.integers(0, 2, size=shape)
    return ((s << 31) | ((e + 127) << 23) | m).astype(np.uint32).view(np.float32)


def test_factor_is_the_one_ulp_difference_of_pam():
    """PAM is piecewise affine in A: moving A one ulp away from zero moves
    A .^ B by the derivative times that step, exactly (the int sum moves by one)."""
    a = normal_values(200000, 1)
    b = normal_values(200000, 2)
    a2 = next_away(a)
    diff = pam_ref.pam_mul_ref(a2, b).astype(np.float64) - pam_ref.pam_mul_ref(a, b).astype(np.float64)
    step = a2.astype(np.float64) - a.astype(np.float64)
    assert np.array_equal(diff, pam_ref.pam_exact_grad_factor(a, b) * step)


def test_factor_against_true_product_for_powers_of_two():
    """When B is a power of two, A .^ B = A * B exactly, whose derivative is B."""
    a = normal_values(50000, 3)
    k = np.random.default_rng(4).integers(-30, 30, size=50000)
    b = (np.where(np.arange(50000) % 2 == 0, 1.0, -1.0) * np.ldexp(1.0, k)).astype(np.float32)
    assert np.array_equal(pam_ref.pam_exact_grad_factor(a, b), b.astype(np.float64))


def test_factor_zero_cases():
    z = np.float32([0.0, -0.0, 1e-40, -1e-41])
    v = np.float32([1.5, -3.0, 2.0 ** -20, 7.0])
    assert np.all(pam_ref.pam_exact_grad_factor(z, v) == 0)
    assert np.all(pam_ref.pam_exact_grad_factor(v, z) == 0)


def test_matrix_grads_are_finite_differences_of_the_product():
    """dX[i,k] and dW[j,k] equal the one-ulp differences of L = sum dY * Y with
    Y the PAM oracle's product, divided by the step (exact rationals in float64:
    every term is a power of two times dY)."""
    g = np.random.default_rng(5)
    t, n, k = 5, 4, 3
    x = normal_values((t, k), 6, -8, 8)
    w = normal_values((n, k), 7, -8, 8)
    dy = normal_values((t, n), 8, -8, 8)
    dx, _, dw, _ = pam_ref.pam_exact_grads_ref(dy, x, w)

    def loss(xx, ww):
        c, _ = pam_ref.pam_gemm_ref(xx, ww, False, True)
        return c                                               # [t, n], float64 exact sums of PAM terms

    base = loss(x, w)
    for i in range(t):
        for kk in range(k):
            x2 = x.copy()
            x2[i, kk] = next_away(x[i, kk])
            dl = ((loss(x2, w) - base) * dy.astype(np.float64)).sum()
            assert dl == dx[i, kk] * (np.float64(x2[i, kk]) - np.float64(x[i, kk]))
    for j in range(n):
        for kk in range(k):
            w2 = w.copy()
            w2[j, kk] = next_away(w[j, kk])
            dl = ((loss(x, w2) - base) * dy.astype(np.float64)).sum()
            assert dl == dw[j, kk] * (np.float64(w2[j, kk]) - np.float64(w[j, kk]))


def test_matrix_grads_with_power_of_two_operands_are_matmuls():
    """With W entries +-2^e the product is X W^T exactly, so dX = dY W; with X
    entries +-2^e, dW = dY^T X (float64 matmuls)."""
    g = np.random.default_rng(9)
    x = normal_values((40, 30), 10)
    w = (np.where(g.random((20, 30)) < 0.5, -1.0, 1.0) * np.ldexp(1.0, g.integers(-10, 10, (20, 30)))).astype(np.float32)
    dy = normal_values((40, 20), 11)
    dx, _, _, _ = pam_ref.pam_exact_grads_ref(dy, x, w)
    assert np.allclose(dx, dy.astype(np.float64) @ w.astype(np.float64), rtol=1e-12, atol=0)
    xp = (np.where(g.random((40, 30)) < 0.5, -1.0, 1.0) * np.ldexp(1.0, g.integers(-10, 10, (40, 30)))).astype(np.float32)
    wn = normal_values((20, 30), 12)
    _, _, dw, _ = pam_ref.pam_exact_grads_ref(dy, xp, wn)
    assert np.allclose(dw, dy.astype(np.float64).T @ xp.astype(np.float64), rtol=1e-12, atol=0)


@pytest.mark.parametrize("mistake", ["no_carry", "no_sign", "carry_from_a_only", "exponent_of_a"])
def test_planted_mistakes_are_caught(mistake):
    """Each plausible slip in the factor breaks the finite-difference pin."""
    a = normal_values(20000, 13)
    b = normal_values(20000, 14)

    def factor(a, b):
        ua = a.view(np.uint32).astype(np.int64)
        ub = b.view(np.uint32).astype(np.int64)
        ea, eb = (ua >> 23) & 0xFF, (ub >> 23) & 0xFF
        fa, fb = ua & 0x7FFFFF, ub & 0x7FFFFF
        carry = ((fa + fb) >= (1 << 23)).astype(np.int64)
        if mistake == "no_carry":
            carry = 0 * carry
        if mistake == "carry_from_a_only":
            carry = (fa >= (1 << 22)).astype(np.int64)
        e = (ea if mistake == "exponent_of_a" else eb) - 127 + carry
        sign = 1.0 if mistake == "no_sign" else np.where(ub >> 31 == 1, -1.0, 1.0)
        return sign * np.ldexp(1.0, e)

    a2 = next_away(a)
    diff = pam_ref.pam_mul_ref(a2, b).astype(np.float64) - pam_ref.pam_mul_ref(a, b).astype(np.float64)
    step = a2.astype(np.float64) - a.astype(np.float64)
    assert not np.array_equal(diff, factor(a, b) * step)
