"""Checks that pin a PAM implementation to what the paper fixes.

Every check takes the implementation under test as an argument, so that the
same checks run on the oracle (tests/test_oracle_pins.py), on deliberately
broken copies of it (tests/test_oracle_mutations.py) and on the C oracle.

  mul(a, b)            float32 arrays -> float32 array (elementwise PAM)
  gemm(A, B, ta, tb)   float32 matrices -> float64 C (sum of PAM terms)

A check returns None when it passes and raises AssertionError otherwise.
None of these checks computes PAM itself; each one compares against true
multiplication, a closed form, or a value the paper prints.
"""
from __future__ import annotations

import math
import os
from fractions import Fraction

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "pam_examples.txt")

F32_MAX = float(np.finfo(np.float32).max)
MIN_NORMAL = 2.0 ** -126


def bits(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float32).view(np.uint32)


def f32(u) -> np.ndarray:
    return np.asarray(u, dtype=np.uint32).view(np.float32)


def load_golden():
    cases = []
    with open(GOLDEN) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            a, b, e, tag = line.split()[:4]
            cases.append((int(a, 16), int(b, 16), int(e, 16), tag))
    return cases


def normal_range_pairs(n: int, seed: int, lo: int = -40, hi: int = 40):
    """Random float32 pairs whose exponents keep every PAM result normal."""
    g = np.random.default_rng(seed)
    ea = g.integers(lo, hi, size=n)
    eb = g.integers(lo, hi, size=n)
    ma = g.integers(0, 1 << 23, size=n)
    mb = g.integers(0, 1 << 23, size=n)
    sa = g.integers(0, 2, size=n)
    sb = g.integers(0, 2, size=n)
    a = ((sa << 31) | ((ea + 127) << 23) | ma).astype(np.uint32).view(np.float32)
    b = ((sb << 31) | ((eb + 127) << 23) | mb).astype(np.uint32).view(np.float32)
    return a, b


# ---------------------------------------------------------------------------
# Scalar pins
# ---------------------------------------------------------------------------

def check_golden(mul):
    """Worked examples printed in, or derived by hand from, Secs. 2.2 and 2.7."""
    cases = load_golden()
    a = f32([c[0] for c in cases])
    b = f32([c[1] for c in cases])
    want = np.array([c[2] for c in cases], dtype=np.uint32)
    got = bits(mul(a, b))
    bad = [cases[i][3] for i in np.nonzero(got != want)[0]]
    assert not bad, f"golden cases differ: {bad}"


def check_max_error_example(mul):
    """Sec. 2.7: relative error at 1.5 .^ 1.5 is exactly -1/9."""
    p = float(mul(np.float32([1.5]), np.float32([1.5]))[0])
    assert Fraction(p) / Fraction(9, 4) - 1 == Fraction(-1, 9)


def check_powers_of_two_exact(mul, n: int = 20000, seed: int = 1):
    """Sec. 2.7: PAM is exact when either operand is a power of two."""
    g = np.random.default_rng(seed)
    a, _ = normal_range_pairs(n, seed)
    k = g.integers(-40, 41, size=n)
    s = np.where(g.random(n) < 0.5, 1.0, -1.0)
    p2 = (s * np.ldexp(1.0, k)).astype(np.float32)
    want = (a.astype(np.float64) * p2.astype(np.float64)).astype(np.float32)
    assert np.array_equal(bits(mul(a, p2)), bits(want)), "power-of-two product not exact (right operand)"
    assert np.array_equal(bits(mul(p2, a)), bits(want)), "power-of-two product not exact (left operand)"
    one = np.ones_like(a)
    assert np.array_equal(bits(mul(a, one)), bits(a)), "pam(a, 1) != a"
    assert np.array_equal(bits(mul(a, -one)), bits(-a)), "pam(a, -1) != -a"


def check_error_bounds(mul, n: int = 50000, seed: int = 2):
    """Secs. 2.2 and 2.7: (8/9)|ab| <= |a .^ b| <= |ab| with the sign of ab.

    From the definition, (1+M_A)(1+M_B) - (1+M_A+M_B) = M_A M_B >= 0 without
    carry and (1+M_A)(1+M_B) - 2(M_A+M_B) = (1-M_A)(1-M_B) >= 0 with carry;
    the ratio is smallest (8/9) at M_A = M_B = 1/2.
    """
    a, b = normal_range_pairs(n, seed)
    ab = a.astype(np.float64) * b.astype(np.float64)        # exact in float64
    p = mul(a, b).astype(np.float64)
    assert np.all(np.sign(p) == np.sign(ab)), "sign differs from the true product"
    r = p / ab
    assert np.all(r <= 1.0), "PAM exceeds the true product in magnitude"
    assert np.all(r >= 8.0 / 9.0), "PAM below 8/9 of the true product"


def check_value_form(mul, n: int = 30000, seed: int = 3):
    """Sec. 2.3: A .^ B = paexp2(palog2 A + palog2 B) for A, B > 0.

    palog2(A) = E_A + M_A and paexp2(x) = 2^floor(x) (1 + x - floor(x)),
    evaluated with frexp/ldexp in float64, where they are exact.
    """
    a, b = normal_range_pairs(n, seed)
    a = np.abs(a)
    b = np.abs(b)

    def palog2(x):
        m, e = np.frexp(x.astype(np.float64))
        return (e - 1) + (2.0 * m - 1.0)

    x = palog2(a) + palog2(b)
    fl = np.floor(x)
    want = np.ldexp(1.0 + (x - fl), fl.astype(np.int64)).astype(np.float32)
    got = mul(a, b)
    assert np.array_equal(bits(got), bits(want)), "bit form differs from paexp2(palog2 + palog2)"


def check_mantissa_grid(mul, mbits: int = 7):
    """Fig. 2 region [1, 2)^2 and its octaves, brute force over all pairs.

    Every pair of mbits-bit mantissas, over a grid of exponents that includes
    the underflow and overflow boundaries, against the value form evaluated
    with exact rationals on a sample and float64 everywhere.
    """
    fr = np.arange(1 << mbits, dtype=np.int64) << (23 - mbits)
    exps = [-126, -100, -64, -63, -62, -1, 0, 1, 63, 64, 65, 100, 127]
    for ea in exps:
        for eb in exps:
            fa, fb = np.meshgrid(fr, fr, indexing="ij")
            fa = fa.reshape(-1)
            fb = fb.reshape(-1)
            a = (((ea + 127) << 23) | fa).astype(np.uint32).view(np.float32)
            b = (((eb + 127) << 23) | fb).astype(np.uint32).view(np.float32)
            # value form with R4 (flush below 2^-126) and R5 (saturate at FLT_MAX)
            x = (ea + fa / 2.0 ** 23) + (eb + fb / 2.0 ** 23)
            fl = np.floor(x)
            v = np.ldexp(1.0 + (x - fl), fl.astype(np.int64))
            v = np.where(v < MIN_NORMAL, 0.0, np.where(v > F32_MAX, F32_MAX, v))
            got = mul(a, b).astype(np.float64)
            assert np.array_equal(got, v), f"mantissa grid differs at exponents ({ea}, {eb})"
    # exact rational spot check of the value form itself on one octave
    for fa in (0, 1, 37, 64, 100, 127):
        for fb in (0, 5, 64, 90, 127):
            ma = Fraction(fa, 1 << mbits)
            mb = Fraction(fb, 1 << mbits)
            s = ma + mb
            want = 2 * s if s >= 1 else 1 + s          # 2^1 (1 + s - 1) or 2^0 (1 + s)
            got = Fraction(float(mul(np.float32([1 + float(ma)]), np.float32([1 + float(mb)]))[0]))
            assert got == want, f"mantissa pair ({fa}, {fb}) differs from the definition"


def check_symmetries(mul, n: int = 20000, seed: int = 4):
    """Commutativity, odd symmetry in each operand, octave periodicity (Fig. 2)."""
    a, b = normal_range_pairs(n, seed, -30, 30)
    p = bits(mul(a, b))
    assert np.array_equal(p, bits(mul(b, a))), "not commutative"
    assert np.array_equal(p ^ np.uint32(0x80000000), bits(mul(-a, b))), "pam(-a, b) != -pam(a, b)"
    assert np.array_equal(p ^ np.uint32(0x80000000), bits(mul(a, -b))), "pam(a, -b) != -pam(a, b)"
    two_a = (a.astype(np.float64) * 2).astype(np.float32)
    assert np.array_equal(bits(mul(two_a, b)), bits((mul(a, b).astype(np.float64) * 2).astype(np.float32))), \
        "pam(2a, b) != 2 pam(a, b)"


def check_monotone(mul, seed: int = 5):
    """For fixed b > 0, a -> pam(a, b) is non-decreasing (piecewise affine, continuous)."""
    g = np.random.default_rng(seed)
    a = np.sort(g.uniform(0.1, 100.0, size=5000)).astype(np.float32)
    for bv in (0.3, 1.0, 1.5, 1.999, 7.25):
        p = mul(a, np.full_like(a, bv)).astype(np.float64)
        assert np.all(np.diff(p) >= 0), f"not monotone for b = {bv}"


def check_range_readings(mul):
    """Underflow / overflow / zero / denormal / NaN / inf readings (Sec. 2.2 prose).

    Sec. 2.2 says the exponent is clamped on under/overflow, denormals may be
    flushed and NaN/inf are handled explicitly; the exact values below follow
    the readings stated in the oracle's header.
    """
    cases = [
        # underflow boundary: 1.5*2^-64 .^ 1.5*2^-63 = 2^-126 exactly (carry)
        (0x1FC00000, 0x20400000, 0x00800000),
        # 1.25*2^-64 .^ 1.25*2^-63 has exponent field 0 -> flushed to +0
        (0x1FA00000, 0x20200000, 0x00000000),
        # 2^-63 .^ 2^-63 = 2^-126 (min normal)
        (0x20000000, 0x20000000, 0x00800000),
        # 2^-64 .^ 2^-63 = 2^-127 -> underflow -> +0; negative sign kept
        (0x1F800000, 0x20000000, 0x00000000),
        (0x9F800000, 0x20000000, 0x80000000),
        # 2^-100 .^ 2^-30 -> +0
        (0x0D800000, 0x30800000, 0x00000000),
        # overflow: 2^64 .^ 2^64 = 2^128 -> FLT_MAX; sign kept
        (0x5F800000, 0x5F800000, 0x7F7FFFFF),
        (0xDF800000, 0x5F800000, 0xFF7FFFFF),
        # FLT_MAX .^ 0.5 = FLT_MAX / 2 exactly (power of two)
        (0x7F7FFFFF, 0x3F000000, 0x7EFFFFFF),
        # largest finite result without overflow: 2^127 .^ 1.99999988 = just below FLT_MAX
        (0x7F000000, 0x3FFFFFFF, 0x7F7FFFFF),
        # zeros and denormals in -> signed zero
        (0x00000000, 0x3F800000, 0x00000000),
        (0x80000000, 0x3F800000, 0x80000000),
        (0x00000000, 0xBF800000, 0x80000000),
        (0x007FFFFF, 0x7F7FFFFF, 0x00000000),
        (0x807FFFFF, 0x3F800000, 0x80000000),
        (0x00000001, 0x7F000000, 0x00000000),
        # inf
        (0x7F800000, 0x3F800000, 0x7F800000),
        (0x7F800000, 0xBF800000, 0xFF800000),
        (0xFF800000, 0xFF800000, 0x7F800000),
        (0x7F800000, 0x00000000, 0x7FC00000),
        (0x7F800000, 0x00000001, 0x7FC00000),
        (0x80000000, 0xFF800000, 0x7FC00000),
        (0x7F800000, 0x00800000, 0x7F800000),
        # NaN in -> canonical quiet NaN
        (0x7FC00000, 0x3F800000, 0x7FC00000),
        (0x7F800001, 0x3F800000, 0x7FC00000),
        (0xFFFFFFFF, 0x00000000, 0x7FC00000),
        (0x3F800000, 0x7FFFFFFF, 0x7FC00000),
        (0x7F800000, 0x7FC00000, 0x7FC00000),
    ]
    a = f32([c[0] for c in cases])
    b = f32([c[1] for c in cases])
    want = np.array([c[2] for c in cases], dtype=np.uint32)
    got = bits(mul(a, b))
    bad = [(hex(c[0]), hex(c[1]), hex(int(g)), hex(c[2])) for c, g in zip(cases, got) if int(g) != c[2]]
    assert not bad, f"range readings differ (a, b, got, want): {bad}"


def check_never_exceeds_true_product(mul, seed: int = 6):
    """|pam(a, b)| <= |a b| over random finite encodings of every class (R4, R5)."""
    g = np.random.default_rng(seed)
    u = g.integers(0, 1 << 32, size=(2, 40000), dtype=np.uint64).astype(np.uint32)
    a = u[0].view(np.float32)
    b = u[1].view(np.float32)
    fin = np.isfinite(a) & np.isfinite(b)
    a = a[fin]
    b = b[fin]
    p = np.abs(mul(a, b).astype(np.float64))
    ab = np.abs(a.astype(np.float64) * b.astype(np.float64))
    assert np.all(p <= ab), "|pam| exceeds |ab|"


SCALAR_CHECKS = [
    check_golden,
    check_max_error_example,
    check_powers_of_two_exact,
    check_error_bounds,
    check_value_form,
    check_mantissa_grid,
    check_symmetries,
    check_monotone,
    check_range_readings,
    check_never_exceeds_true_product,
]


# ---------------------------------------------------------------------------
# Matrix-product pins
# ---------------------------------------------------------------------------

def _opnd(x, trans):
    return np.ascontiguousarray(x.T) if trans else x


def check_gemm_identity(gemm, seed: int = 10):
    """op(B) = I: every output is one term pam(a, 1) = a plus exact zeros."""
    g = np.random.default_rng(seed)
    for ta in (False, True):
        for tb in (False, True):
            a_op = g.standard_normal((7, 5)).astype(np.float32)
            eye = np.eye(5, dtype=np.float32)
            c = gemm(_opnd(a_op, ta), _opnd(eye, tb), ta, tb)
            assert np.array_equal(c, a_op.astype(np.float64)), f"identity product differs (ta={ta}, tb={tb})"


def check_gemm_outer(gemm, mul, seed: int = 11):
    """K = 1: C = elementwise PAM of the broadcast column and row."""
    g = np.random.default_rng(seed)
    col = g.standard_normal((9, 1)).astype(np.float32)
    row = g.standard_normal((1, 6)).astype(np.float32)
    c = gemm(col, row, False, False)
    want = mul(np.repeat(col, 6, axis=1), np.repeat(row, 9, axis=0)).astype(np.float64)
    assert np.array_equal(c, want), "K = 1 product differs from elementwise PAM"


def check_gemm_powers_of_two(gemm, seed: int = 12):
    """op(B) entries +-2^k: every PAM term is exact, so C = op(A) op(B) (float64 matmul)."""
    g = np.random.default_rng(seed)
    for (m, n, k) in ((13, 11, 17), (8, 8, 8)):
        for ta in (False, True):
            for tb in (False, True):
                a_op = g.standard_normal((m, k)).astype(np.float32)
                e = g.integers(-6, 7, size=(k, n))
                s = np.where(g.random((k, n)) < 0.5, 1.0, -1.0)
                b_op = (s * np.ldexp(1.0, e)).astype(np.float32)
                c = gemm(_opnd(a_op, ta), _opnd(b_op, tb), ta, tb)
                want = a_op.astype(np.float64) @ b_op.astype(np.float64)
                assert np.allclose(c, want, rtol=1e-12, atol=1e-12), \
                    f"power-of-two product differs ({m}x{n}x{k}, ta={ta}, tb={tb})"


def check_gemm_nonneg_bounds(gemm, seed: int = 13):
    """A, B >= 0: (8/9) AB <= C <= AB elementwise (per-term bound, Sec. 2.7)."""
    g = np.random.default_rng(seed)
    a = g.uniform(0.01, 3.0, size=(8, 10)).astype(np.float32)
    b = g.uniform(0.01, 3.0, size=(10, 12)).astype(np.float32)
    c = gemm(a, b, False, False)
    ab = a.astype(np.float64) @ b.astype(np.float64)
    assert np.all(c <= ab * (1 + 1e-12)), "C exceeds AB"
    assert np.all(c >= ab * (8.0 / 9.0) * (1 - 1e-12)), "C below (8/9) AB"


def check_gemm_bruteforce(gemm, seed: int = 14):
    """Tiny product by definition: Python loops, value form, exact rationals."""
    g = np.random.default_rng(seed)
    m, n, k = 3, 4, 5
    a = g.standard_normal((m, k)).astype(np.float32)
    b = g.standard_normal((k, n)).astype(np.float32)

    def pam_exact(x: float, y: float) -> Fraction:
        # Sec. 2.2 with A = (-1)^S 2^E (1 + M), exponents from frexp
        mx, ex = math.frexp(abs(x))
        my, ey = math.frexp(abs(y))
        ma = Fraction(mx) * 2 - 1
        mb = Fraction(my) * 2 - 1
        carry = 1 if ma + mb >= 1 else 0
        v = Fraction(2) ** ((ex - 1) + (ey - 1) + carry) * (1 + ma + mb - carry)
        return -v if (x < 0) != (y < 0) else v

    for ta in (False, True):
        for tb in (False, True):
            c = gemm(_opnd(a, ta), _opnd(b, tb), ta, tb)
            for i in range(m):
                for j in range(n):
                    want = sum((pam_exact(float(a[i, kk]), float(b[kk, j])) for kk in range(k)), Fraction(0))
                    assert abs(Fraction(float(c[i, j])) - want) <= abs(want) * Fraction(1, 1 << 50), \
                        f"brute-force entry ({i},{j}) differs (ta={ta}, tb={tb})"


def check_gemm_zero_rows(gemm, seed: int = 15):
    """A zero row of op(A) (or denormal-only) gives an exactly zero output row."""
    g = np.random.default_rng(seed)
    a = g.standard_normal((4, 6)).astype(np.float32)
    a[1, :] = 0.0
    a[2, :] = np.float32(1e-40)                                   # denormals
    b = g.standard_normal((6, 5)).astype(np.float32)
    c = gemm(a, b, False, False)
    assert np.all(c[1] == 0) and np.all(c[2] == 0), "zero / denormal row does not give zeros"


GEMM_CHECKS = [
    check_gemm_identity,
    check_gemm_powers_of_two,
    check_gemm_nonneg_bounds,
    check_gemm_bruteforce,
    check_gemm_zero_rows,
]
