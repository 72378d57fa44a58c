"""The exact derivative of PAM products (Table 1, reading R15), pinned by
one-ulp finite differences of the PAM oracle itself (bit form, Sec. 2.2) and
of the unclamped value form (Sec. 2.3), over every pair of exponent fields --
the underflow and saturation regions and their boundaries included -- by
true multiplication where one operand is a power of two, by the identity
A .^ 1 = A, by the zero cases, and, for the matrix form, by finite
differences of the PAM product and by PAM of dY with the power of two
(Sec. "Derivatives": that product is performed exactly by PAM, which reads a
denormal dY as zero).  Planted mistakes in every branch of the reading are
each caught by one of these pins."""
import numpy as np
import pytest

from oracle import pam_ref

FLT_MAX = float(np.finfo(np.float32).max)
TINY = 2.0 ** -126


def next_away(x):
    """The float32 one ulp further from zero (+-inf beyond +-FLT_MAX)."""
    x = np.asarray(x, np.float32)
    with np.errstate(over="ignore"):
        return np.nextafter(x, np.where(x < 0, np.float32(-np.inf), np.float32(np.inf)).astype(np.float32))


def normal_values(shape, seed, lo=-20, hi=20):
    g = np.random.default_rng(seed)
    e = g.integers(lo, hi, size=shape)
    m = g.integers(0, 1 << 23, size=shape)
    s = g.integers(0, 2, size=shape)
    return ((s << 31) | ((e + 127) << 23) | m).astype(np.uint32).view(np.float32)


def all_exponent_pairs(seed, per_pair=3):
    """Operands with every pair of exponent fields 1..254, random mantissas
    and signs; the last A of each pair has an all-ones mantissa (the next ulp
    changes binade) and one B a zero mantissa."""
    g = np.random.default_rng(seed)
    ea, eb = np.meshgrid(np.arange(1, 255), np.arange(1, 255), indexing="ij")
    ea = np.repeat(ea.reshape(-1), per_pair)
    eb = np.repeat(eb.reshape(-1), per_pair)
    n = ea.size
    ma = g.integers(0, 1 << 23, size=n)
    mb = g.integers(0, 1 << 23, size=n)
    ma[per_pair - 1::per_pair] = (1 << 23) - 1
    mb[0::per_pair] = 0
    sa = g.integers(0, 2, size=n)
    sb = g.integers(0, 2, size=n)
    a = ((sa << 31) | (ea << 23) | ma).astype(np.uint32).view(np.float32)
    b = ((sb << 31) | (eb << 23) | mb).astype(np.uint32).view(np.float32)
    return a, b


def unclamped_value(a, b):
    """|A .^ B| before any range handling, in float64, from the value form of
    Sec. 2.3: paexp2(palog2|A| + palog2|B|), exact for float32 operands.
    palog2 of a normal x = 2^E (1 + M) is E + M; paexp2(y) = 2^floor(y) (1 + y - floor(y))."""
    def palog2(x):
        m, e = np.frexp(np.abs(np.asarray(x, np.float64)))          # |x| = m 2^e, m in [1/2, 1)
        return (e - 1) + (2.0 * m - 1.0)
    y = palog2(a) + palog2(b)
    fl = np.floor(y)
    return np.ldexp(1.0 + (y - fl), fl.astype(np.int64))


def regime(a, b):
    """-1: A .^ B underflows (R4), 1: it saturates (R5), 0: not clamped."""
    u = unclamped_value(a, b)
    return np.where(u < TINY, -1, np.where(u > FLT_MAX, 1, 0))


# ---------------------------------------------------------------------------
# Pins, each a function of the factor (and of the matrix-form reference), so
# that planted mistakes can be run through them.
# ---------------------------------------------------------------------------

def pin_bit_form_differences(factor):
    """Over every exponent pair: where A and A one ulp further from zero lie in
    the same regime (both clamped the same way, or neither), the one-ulp
    difference of the bit-form PAM is the derivative times the step (exact:
    every quantity is a float32 value or a power-of-two multiple of one).
    Clamped pairs then have a zero difference: the flat regions."""
    a, b = all_exponent_pairs(21)
    a2 = next_away(a)
    fin = np.isfinite(a2)
    a, b, a2 = a[fin], b[fin], a2[fin]
    same = regime(a, b) == regime(a2, b)
    a, b, a2 = a[same], b[same], a2[same]
    diff = pam_ref.pam_mul_ref(a2, b).astype(np.float64) - pam_ref.pam_mul_ref(a, b).astype(np.float64)
    step = a2.astype(np.float64) - a.astype(np.float64)
    got = np.asarray(factor(a, b), np.float64) * step
    r = regime(a, b)
    # every regime must be exercised in bulk
    assert (r == -1).sum() > 20000 and (r == 1).sum() > 20000 and (r == 0).sum() > 100000
    bad = got != diff
    assert not bad.any(), (f"{int(bad.sum())} pairs differ, e.g. a={a[bad][0]!r} b={b[bad][0]!r}: "
                           f"{got[bad][0] / step[bad][0]!r} vs difference quotient {diff[bad][0] / step[bad][0]!r}")


def boundary_pairs(seed):
    """Pairs whose magnitude sum |A| + |B| - bias lands on, or one ulp beside,
    the underflow boundary 0x00800000 and the saturation boundary 0x7F7FFFFF,
    over many exponent splits."""
    g = np.random.default_rng(seed)
    out_a, out_b = [], []
    for target in (0x00800000 - 1, 0x00800000, 0x00800000 + 1, 0x7F7FFFFF - 1, 0x7F7FFFFF, 0x7F7FFFFF + 1):
        for _ in range(4000):
            mb = int(g.integers(0x00800000, 0x7F800000))
            ma = target + 0x3F800000 - mb
            if not 0x00800000 <= ma < 0x7F800000:
                continue
            out_a.append(ma | (int(g.integers(0, 2)) << 31))
            out_b.append(mb | (int(g.integers(0, 2)) << 31))
    return (np.array(out_a, np.uint32).view(np.float32), np.array(out_b, np.uint32).view(np.float32))


def pin_boundaries_by_value_form(factor):
    """On the clamp boundaries, independently of the bit form: a clamped
    product (value form below 2^-126 or above FLT_MAX) has derivative 0; an
    unclamped one has the slope of the unclamped value form as |A| grows by
    one ulp (times sgn(B))."""
    a, b = boundary_pairs(22)
    a2 = next_away(a)
    keep = np.isfinite(a2)
    a, b, a2 = a[keep], b[keep], a2[keep]
    r = regime(a, b)
    assert (r == -1).sum() > 1000 and (r == 1).sum() > 1000 and (r == 0).sum() > 1000
    slope = (unclamped_value(a2, b) - unclamped_value(a, b)) / (np.abs(a2.astype(np.float64)) -
                                                                np.abs(a.astype(np.float64)))
    want = np.where(r == 0, np.sign(b.astype(np.float64)) * slope, 0.0)
    got = np.asarray(factor(a, b), np.float64)
    bad = got != want
    assert not bad.any(), f"{int(bad.sum())} boundary pairs differ, e.g. a={a[bad][0]!r} b={b[bad][0]!r}"


def pin_identity_and_powers_of_two(factor):
    """A .^ (+-1) = +-A for every normal A (FLT_MAX and 2^-126 included), so
    the derivative is +-1; A .^ 2^k = A 2^k exactly, so the derivative is 2^k
    where A 2^k is a normal float32 and 0 where the product is clamped."""
    a = np.concatenate([normal_values(40000, 23, -126, 128),
                        np.float32([FLT_MAX, -FLT_MAX, TINY, -TINY, 1.0, -1.0])])
    for one in (1.0, -1.0):
        assert np.array_equal(np.asarray(factor(a, np.full_like(a, one)), np.float64), np.full(a.size, one))
    g = np.random.default_rng(24)
    k = g.integers(-126, 128, size=a.size)
    b = (np.where(g.random(a.size) < 0.5, -1.0, 1.0) * np.ldexp(1.0, k)).astype(np.float32)
    prod = np.abs(a.astype(np.float64) * b.astype(np.float64))
    want = np.where((prod < TINY) | (prod > FLT_MAX), 0.0, b.astype(np.float64))
    assert np.array_equal(np.asarray(factor(a, b), np.float64), want)


def pin_zero_operands(factor):
    z = np.float32([0.0, -0.0, 1e-40, -1e-41, 2.0 ** -149])
    v = np.float32([1.5, -3.0, 2.0 ** -20, 7.0, FLT_MAX])
    assert np.all(np.asarray(factor(z, v)) == 0)
    assert np.all(np.asarray(factor(v, z)) == 0)


def pin_unchanged_sign_of_a(factor):
    """d(A .^ B)/dA does not depend on the sign of A (|A .^ B| grows with |A|,
    the sign is S_A + S_B): the one-ulp difference pins, run on -A."""
    a = normal_values(20000, 25)
    b = normal_values(20000, 26)
    assert np.array_equal(np.asarray(factor(a, b)), np.asarray(factor(-a, b)))


FACTOR_PINS = [pin_bit_form_differences, pin_boundaries_by_value_form, pin_identity_and_powers_of_two,
               pin_zero_operands, pin_unchanged_sign_of_a]


@pytest.mark.parametrize("pin", FACTOR_PINS, ids=lambda f: f.__name__)
def test_factor_pins(pin):
    pin(pam_ref.pam_exact_grad_factor)


def test_flat_region_examples():
    """The examples of the flat regions: 2^-100 .^ 2^-30 underflows and
    2^100 .^ 2^40 saturates, so moving A changes nothing; 1.5 2^127 .^ 1.75
    saturates too (the carry takes its exponent past 127)."""
    a = np.float32([2.0 ** -100, 2.0 ** 100, 1.5 * 2.0 ** 127, 2.0 ** -63])
    b = np.float32([2.0 ** -30, 2.0 ** 40, 1.75, 2.0 ** -63])
    got = pam_ref.pam_exact_grad_factor(a, b)
    assert got.tolist() == [0.0, 0.0, 0.0, 2.0 ** -63]


# ---------------------------------------------------------------------------
# Matrix form
# ---------------------------------------------------------------------------

def fd_case(kind):
    """(dy, x, w) for the matrix finite-difference pin.  Exponent ranges are
    chosen so that every float64 sum involved is exact (terms within a
    narrow band), while whole rows of X sit in the clamp regions:
      narrow     X, W, dY ~ 2^[-8, 8];
      underflow  X row 0 ~ 2^[-100, -95], W ~ 2^[-38, -32]: every product of
                 that row underflows (R4), the other rows' do not;
      saturate   X row 0 ~ 2^[100, 105], W ~ 2^[30, 35]: every product of
                 that row saturates (R5)."""
    t, n, k = 5, 4, 3
    wr = {"narrow": (-8, 8), "underflow": (-38, -32), "saturate": (30, 35)}[kind]
    x = normal_values((t, k), 6, -8, 8)
    if kind == "underflow":
        x[0] = normal_values(k, 30, -100, -95)
    if kind == "saturate":
        x[0] = normal_values(k, 31, 100, 105)
    w = normal_values((n, k), 7, *wr)
    dy = normal_values((t, n), 8, -8, 8)
    return dy, x, w


def pin_matrix_finite_differences(grads):
    """dX[i,k] and dW[j,k] equal the one-ulp differences of L = sum dY * Y with
    Y the PAM oracle's product, divided by the step (exact rationals in float64:
    every term is a power of two times dY); rows whose products are clamped
    have zero derivatives, as their products do not move."""
    for kind in ("narrow", "underflow", "saturate"):
        dy, x, w = fd_case(kind)
        t, k = x.shape
        n = w.shape[0]
        dx, _, dw, _ = grads(dy, x, w)

        def loss(xx, ww):
            c, _ = pam_ref.pam_gemm_ref(xx, ww, False, True)
            return c

        base = loss(x, w)
        for i in range(t):
            for kk in range(k):
                x2 = x.copy()
                x2[i, kk] = next_away(x[i, kk])
                dl = ((loss(x2, w) - base) * dy.astype(np.float64)).sum()
                assert dl == dx[i, kk] * (np.float64(x2[i, kk]) - np.float64(x[i, kk])), (kind, "dX", i, kk)
        for j in range(n):
            for kk in range(k):
                w2 = w.copy()
                w2[j, kk] = next_away(w[j, kk])
                dl = ((loss(x, w2) - base) * dy.astype(np.float64)).sum()
                assert dl == dw[j, kk] * (np.float64(w2[j, kk]) - np.float64(w[j, kk])), (kind, "dW", j, kk)
        if kind != "narrow":
            assert np.all(dx[0] == 0.0), kind


def pin_terms_are_pam_of_dy(grads):
    """Each term dY * g is the PAM of dY and the power of two g (exact there,
    Sec. 2.7), so a denormal or zero dY contributes nothing: dX summed from
    pam(dY[i,j], g) in increasing j, with g taken from B = W's one-operand
    case W = +-2^e (g = W wherever X .^ W is not clamped)."""
    g = np.random.default_rng(27)
    t, n, k = 30, 20, 10
    x = normal_values((t, k), 28, -10, 10)
    w = (np.where(g.random((n, k)) < 0.5, -1.0, 1.0) * np.ldexp(1.0, g.integers(-5, 5, (n, k)))).astype(np.float32)
    dy = normal_values((t, n), 29, -10, 10)
    flat = dy.reshape(-1)
    idx = g.choice(flat.size, size=120, replace=False)
    flat[idx[:40]] = np.float32(1e-40)
    flat[idx[40:80]] = np.float32(-3e-39)
    flat[idx[80:]] = np.float32(0.0)
    dy[0] = np.float32(2.0 ** -130)        # a row of denormal dY alone: its dX row is exactly zero
    dy[1, ::2] = np.float32(-1e-39)
    dx, _, _, _ = grads(dy, x, w)
    assert np.all(dx[0] == 0.0)
    want = np.zeros((t, k))
    for j in range(n):
        want += pam_ref.pam_mul_ref(dy[:, j:j + 1], w[j:j + 1, :]).astype(np.float64)
    assert np.array_equal(dx, want)


def pin_power_of_two_operands_are_matmuls(grads):
    """With W entries +-2^e the product is X W^T exactly, so dX = dY W; with X
    entries +-2^e, dW = dY^T X (float64 matmuls)."""
    g = np.random.default_rng(9)
    x = normal_values((40, 30), 10)
    w = (np.where(g.random((20, 30)) < 0.5, -1.0, 1.0) * np.ldexp(1.0, g.integers(-10, 10, (20, 30)))).astype(np.float32)
    dy = normal_values((40, 20), 11)
    dx, _, _, _ = grads(dy, x, w)
    assert np.allclose(dx, dy.astype(np.float64) @ w.astype(np.float64), rtol=1e-12, atol=0)
    xp = (np.where(g.random((40, 30)) < 0.5, -1.0, 1.0) * np.ldexp(1.0, g.integers(-10, 10, (40, 30)))).astype(np.float32)
    wn = normal_values((20, 30), 12)
    _, _, dw, _ = grads(dy, xp, wn)
    assert np.allclose(dw, dy.astype(np.float64).T @ xp.astype(np.float64), rtol=1e-12, atol=0)


GRAD_PINS = [pin_matrix_finite_differences, pin_terms_are_pam_of_dy, pin_power_of_two_operands_are_matmuls]


@pytest.mark.parametrize("pin", GRAD_PINS, ids=lambda f: f.__name__)
def test_grad_pins(pin):
    pin(pam_ref.pam_exact_grads_ref)


# ---------------------------------------------------------------------------
# Planted mistakes: every branch of R15 mutated, each caught by some pin.
# ---------------------------------------------------------------------------

def mutant_factor(mistake):
    def factor(a, b):
        a = np.asarray(a, np.float32)
        b = np.asarray(b, np.float32)
        ua = a.view(np.uint32).astype(np.int64)
        ub = b.view(np.uint32).astype(np.int64)
        ea, eb = (ua >> 23) & 0xFF, (ub >> 23) & 0xFF
        fa, fb = ua & 0x7FFFFF, ub & 0x7FFFFF
        carry = ((fa + fb) >= (1 << 23)).astype(np.int64)
        if mistake == "no_carry":
            carry = 0 * carry
        if mistake == "carry_from_a_only":
            carry = (fa >= (1 << 22)).astype(np.int64)
        if mistake == "carry_strict":
            carry = ((fa + fb) > (1 << 23)).astype(np.int64)
        e = (ea if mistake == "exponent_of_a" else eb) - 127 + carry
        if mistake == "no_sign":
            sign = 1.0
        elif mistake == "sign_of_a":
            sign = np.where(ua >> 31 == 1, -1.0, 1.0)
        elif mistake == "sign_of_product":
            sign = np.where((ua ^ ub) >> 31 == 1, -1.0, 1.0)
        else:
            sign = np.where(ub >> 31 == 1, -1.0, 1.0)
        g = sign * np.ldexp(1.0, e)
        t = (ua & 0x7FFFFFFF) + (ub & 0x7FFFFFFF) - 0x3F800000
        under = t < 0x00800000
        over = t > 0x7F7FFFFF
        if mistake == "formula_in_underflow":
            under = np.zeros_like(under)
        if mistake == "formula_in_saturation":
            over = np.zeros_like(over)
        if mistake == "underflow_off_by_one":
            under = t <= 0x00800000
        if mistake == "saturation_off_by_one":
            over = t >= 0x7F7FFFFF
        if mistake == "range_from_exponents_only":
            e_sum = ea + eb - 254
            under = e_sum < -126
            over = e_sum > 127
        zero = (ea == 0) | (eb == 0)
        if mistake == "denormal_a_kept":
            zero = (ua & 0x7FFFFFFF) == 0
            g = np.where(ea == 0, sign * np.ldexp(1.0, eb - 127), g)
        if mistake == "zero_b_kept":
            zero = ea == 0
        return np.where(zero | under | over, 0.0, g)
    return factor


FACTOR_MISTAKES = ["no_carry", "carry_from_a_only", "carry_strict", "exponent_of_a", "no_sign", "sign_of_a",
                   "sign_of_product", "formula_in_underflow", "formula_in_saturation", "underflow_off_by_one",
                   "saturation_off_by_one", "range_from_exponents_only", "denormal_a_kept", "zero_b_kept"]


def caught(pins, impl):
    for pin in pins:
        try:
            pin(impl)
        except AssertionError:
            return True
    return False


@pytest.mark.parametrize("mistake", FACTOR_MISTAKES)
def test_planted_factor_mistakes_are_caught(mistake):
    assert caught(FACTOR_PINS, mutant_factor(mistake)), mistake


def test_unmutated_factor_copy_passes():
    """The mutation harness itself: with no mistake it agrees with every pin."""
    assert not caught(FACTOR_PINS, mutant_factor("none"))


def mutant_grads(mistake):
    def grads(dy, x, w):
        dy = np.asarray(dy, np.float32)
        if mistake != "denormal_dy_kept":
            dy = np.where(np.abs(dy) < np.float32(TINY), np.float32(0.0), dy)
        dy = dy.astype(np.float64)
        factor = pam_ref.pam_exact_grad_factor
        t, n = dy.shape
        k = x.shape[1]
        dx = np.zeros((t, k))
        dw = np.zeros((n, k))
        for j in range(n):
            if mistake == "dx_operands_swapped":
                gx = factor(w[j:j + 1, :], x)
            else:
                gx = factor(x, w[j:j + 1, :])
            dx += dy[:, j:j + 1] * gx
            gw = factor(x if mistake == "dw_operands_swapped" else w[j:j + 1, :],
                        w[j:j + 1, :] if mistake == "dw_operands_swapped" else x)
            dw[j] = (dy[:, j:j + 1] * gw).sum(axis=0)
        return dx, np.abs(dx), dw, np.abs(dw)
    return grads


@pytest.mark.parametrize("mistake", ["denormal_dy_kept", "dx_operands_swapped", "dw_operands_swapped"])
def test_planted_grad_mistakes_are_caught(mistake):
    assert caught(GRAD_PINS, mutant_grads(mistake)), mistake
