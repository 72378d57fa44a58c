"""Checks that pin PAD, palog2 and paexp2 implementations to what the paper fixes.

Every check takes the implementation under test as an argument (float32 arrays
in, float32 array out), so that the same checks run on the oracle, on
deliberately broken copies of it and on the HIP kernels:

  pad(a, b)    elementwise piecewise affine division (Sec. 2.3)
  palog2(a)    elementwise palog2 (Sec. 2.3)
  paexp2(a)    elementwise paexp2 (Sec. 2.3)

None of these checks computes the operations the way the oracle does: each
compares against exact rationals, true division, log2 / exp2 bounds, the
inverse relation to PAM the paper states, or hand-derived worked examples.
"""
from __future__ import annotations

import math
import os
from fractions import Fraction

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "pa_examples.txt")
QNAN = 0x7FC00000


def bits(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float32).view(np.uint32)


def f32(u) -> np.ndarray:
    return np.asarray(u, dtype=np.uint32).view(np.float32)


def exact(u: int) -> Fraction:
    """Exact value of a finite normal float32 encoding."""
    s, ex, fr = u >> 31, (u >> 23) & 0xFF, u & 0x7FFFFF
    v = (1 + Fraction(fr, 1 << 23)) * Fraction(2) ** (ex - 127)
    return -v if s else v


def load_golden(op: str):
    out = []
    with open(GOLDEN) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            o, a, b, e, tag = line.split()[:5]
            if o == op:
                out.append((int(a, 16), int(b, 16), int(e, 16), tag))
    return out


def normal_pairs(n: int, seed: int, lo: int = -40, hi: int = 40):
    g = np.random.default_rng(seed)
    ea, eb = g.integers(lo, hi, size=n), g.integers(lo, hi, size=n)
    ma, mb = g.integers(0, 1 << 23, size=n), g.integers(0, 1 << 23, size=n)
    sa, sb = g.integers(0, 2, size=n), g.integers(0, 2, size=n)
    a = ((sa << 31) | ((ea + 127) << 23) | ma).astype(np.uint32).view(np.float32)
    b = ((sb << 31) | ((eb + 127) << 23) | mb).astype(np.uint32).view(np.float32)
    return a, b


def is_nearest_even(got_bits: int, q: Fraction) -> bool:
    """got is the float32 nearest to q > 0, ties to even (checked against neighbours)."""
    v = exact(got_bits)
    d = abs(v - q)
    for nb in (got_bits - 1, got_bits + 1):
        if ((nb >> 23) & 0xFF) in (0, 255):
            continue
        dn = abs(exact(nb) - q)
        if dn < d:
            return False
        if dn == d and (got_bits & 1):
            return False
    return True


# ---------------------------------------------------------------------------
# PAD
# ---------------------------------------------------------------------------

def check_pad_golden(pad):
    """Hand-derived examples of Sec. 2.3's PAD lines (R10 borrow)."""
    cases = load_golden("pad")
    got = bits(pad(f32([c[0] for c in cases]), f32([c[1] for c in cases])))
    bad = [c[3] for c, g in zip(cases, got) if int(g) != c[2]]
    assert not bad, f"PAD golden cases differ: {bad}"


def check_pad_inverts_pam(pad, mul):
    """Sec. 2.3: PAD is defined as the inverse of PAM: (a .^ b) ./ b == a."""
    a, b = normal_pairs(20000, 11)
    prod = mul(a, b)
    back = pad(prod, b)
    assert np.array_equal(bits(back), bits(a)), "pad(pam(a, b), b) != a"
    # and the other way round: (a ./ b) .^ b == a
    q = pad(a, b)
    assert np.array_equal(bits(mul(q, b)), bits(a)), "pam(pad(a, b), b) != a"


def check_pad_powers_of_two(pad):
    """Dividing by 2^k only moves the exponent: exact, like true division."""
    g = np.random.default_rng(12)
    a, _ = normal_pairs(4000, 13)
    k = g.integers(-30, 30, size=a.size)
    p2 = np.ldexp(np.float32(1.0), k).astype(np.float32)
    got = pad(a, p2)
    assert np.array_equal(bits(got), bits((a.astype(np.float64) / p2.astype(np.float64)).astype(np.float32)))
    j = g.integers(-60, 60, size=a.size)
    pj = np.ldexp(np.float32(1.0), j).astype(np.float32)
    assert np.array_equal(bits(pad(pj, p2)), bits(np.ldexp(np.float32(1.0), j - k).astype(np.float32)))


def check_pad_bounds(pad):
    """For positive a, b: a/b <= a ./ b <= (9/8) a/b (inverse of 8/9 ab <= a .^ b <= ab)."""
    a, b = normal_pairs(3000, 14)
    a, b = np.abs(a), np.abs(b)
    got = pad(a, b)
    for x, y, z in zip(bits(a), bits(b), bits(got)):
        q = exact(int(x)) / exact(int(y))
        v = exact(int(z))
        assert q <= v <= Fraction(9, 8) * q, (hex(x), hex(y), hex(z))


def check_pad_rational_grid(pad):
    """All 7-bit mantissa pairs over a grid of exponents (including the
    under/overflow edges) against Sec. 2.3's lines evaluated in exact rationals."""
    mant = np.arange(128, dtype=np.int64) << 16
    exps = np.array([1, 2, 60, 126, 127, 128, 190, 253, 254], dtype=np.int64)
    ua = ((exps[:, None] << 23) | mant[None, :]).reshape(-1)
    ua, ub = np.meshgrid(ua, ua, indexing="ij")
    ua, ub = ua.reshape(-1), ub.reshape(-1)
    got = bits(pad(f32(ua), f32(ub))).astype(np.int64)
    for x, y, z in zip(ua[::31], ub[::31], got[::31]):
        ea, fa = (int(x) >> 23) - 127, Fraction(int(x) & 0x7FFFFF, 1 << 23)
        eb, fb = (int(y) >> 23) - 127, Fraction(int(y) & 0x7FFFFF, 1 << 23)
        borrow = 1 if fa < fb else 0
        e = ea - eb - borrow
        m = fa - fb + borrow
        assert 0 <= m < 1
        if e < -126:
            want = 0
        elif e > 127:
            want = 0x7F7FFFFF
        else:
            want = ((e + 127) << 23) | int(m * (1 << 23))
        assert int(z) == want, (hex(x), hex(y), hex(z), hex(want))


def check_pad_symmetries(pad):
    """Sign is S_A - S_B (mod 2); a ./ a = 1; a ./ 1 = a."""
    a, b = normal_pairs(5000, 15)
    p = bits(pad(a, b))
    assert np.array_equal(bits(pad(-a, b)), p ^ 0x80000000)
    assert np.array_equal(bits(pad(a, -b)), p ^ 0x80000000)
    assert np.array_equal(bits(pad(-a, -b)), p)
    absa = np.abs(a)
    assert np.all(pad(absa, absa) == np.float32(1.0))
    assert np.array_equal(bits(pad(a, np.ones_like(a))), bits(a))


def check_pad_specials(pad):
    """Reading R12 (parity pinned by reading, not by the paper)."""
    inf, nan = np.float32(np.inf), np.float32(np.nan)
    den = f32([0x00000005])[0]
    rows = [  # a, b, expected bits
        (0.0, 2.0, 0x00000000), (-0.0, 2.0, 0x80000000), (den, 2.0, 0x00000000),
        (2.0, 0.0, 0x7F800000), (2.0, -0.0, 0xFF800000), (-2.0, den, 0xFF800000),
        (0.0, 0.0, QNAN), (den, -0.0, QNAN), (inf, inf, QNAN), (nan, 1.0, QNAN), (1.0, nan, QNAN),
        (inf, 3.0, 0x7F800000), (-inf, 3.0, 0xFF800000), (inf, 0.0, 0x7F800000),
        (3.0, inf, 0x00000000), (3.0, -inf, 0x80000000), (0.0, inf, 0x00000000),
        (2.0 ** -100, 2.0 ** 40, 0x00000000),            # exponent field <= 0
        (2.0 ** 100, 2.0 ** -40, 0x7F7FFFFF),            # exponent field >= 255
        (1.5 * 2.0 ** -126, 1.5, 0x00800000),            # exactly min normal
    ]
    a = np.array([r[0] for r in rows], dtype=np.float32)
    b = np.array([r[1] for r in rows], dtype=np.float32)
    got = bits(pad(a, b))
    bad = [(float(x), float(y), hex(int(g)), hex(r[2])) for x, y, g, r in zip(a, b, got, rows) if int(g) != r[2]]
    assert not bad, f"PAD special cases differ: {bad}"


PAD_CHECKS = [check_pad_golden, check_pad_powers_of_two, check_pad_bounds, check_pad_rational_grid,
              check_pad_symmetries, check_pad_specials]


# ---------------------------------------------------------------------------
# palog2
# ---------------------------------------------------------------------------

def check_palog2_golden(palog2):
    cases = load_golden("palog2")
    got = bits(palog2(f32([c[0] for c in cases])))
    bad = [c[3] for c, g in zip(cases, got) if int(g) != c[2]]
    assert not bad, f"palog2 golden cases differ: {bad}"


def check_palog2_powers_and_first_octaves(palog2):
    """palog2(2^k) = k; palog2(1 + M) = M and palog2((1 + M) / 2) = M - 1 exactly."""
    k = np.arange(-126, 128)
    got = palog2(np.ldexp(np.float32(1.0), k).astype(np.float32))
    assert np.array_equal(got, k.astype(np.float32))
    g = np.random.default_rng(21)
    m = g.integers(0, 1 << 23, size=20000)
    x = (0x3F800000 | m).astype(np.uint32).view(np.float32)
    assert np.array_equal(palog2(x).astype(np.float64), m / float(1 << 23))
    xh = (0x3F000000 | m).astype(np.uint32).view(np.float32)
    assert np.array_equal(palog2(xh).astype(np.float64), m / float(1 << 23) - 1.0)


def check_palog2_nearest(palog2):
    """Elsewhere E + M needs up to 31 bits: the result is the nearest float32 (R13)."""
    a, _ = normal_pairs(3000, 22, lo=-126, hi=128)
    a = np.abs(a)
    got = bits(palog2(a))
    for x, z in zip(bits(a), got):
        ex, fr = (int(x) >> 23) - 127, int(x) & 0x7FFFFF
        q = Fraction(ex) + Fraction(fr, 1 << 23)
        if q == 0:
            assert int(z) == 0
            continue
        zb = int(z)
        assert (zb >> 31) == (1 if q < 0 else 0), hex(x)
        assert is_nearest_even(zb & 0x7FFFFFFF, abs(q)), (hex(x), hex(zb))


def check_palog2_mitchell_bounds(palog2):
    """log2(1 + M) - 0.0861 <= M <= log2(1 + M): palog2 sits just below log2."""
    a, _ = normal_pairs(20000, 23, lo=-100, hi=100)
    a = np.abs(a)
    got = palog2(a).astype(np.float64)
    ref = np.log2(a.astype(np.float64))
    slack = np.abs(ref) * 2.0 ** -23 + 1e-12          # one float32 rounding of the result
    assert np.all(got <= ref + slack)
    assert np.all(got >= ref - 0.086072 - slack)


def check_palog2_monotone(palog2):
    u = np.sort(np.random.default_rng(24).integers(0x00800000, 0x7F800000, size=50000)).astype(np.uint32)
    got = palog2(u.view(np.float32)).astype(np.float64)
    assert np.all(got[1:] >= got[:-1])


def check_palog2_specials(palog2):
    """Reading R13 (parity pinned by reading)."""
    rows = [(0x00000000, 0xFF800000), (0x80000000, 0xFF800000), (0x00000007, 0xFF800000),
            (0xBF800000, QNAN), (0xFF800000, QNAN), (0x7F800000, 0x7F800000), (0x7FC00001, QNAN),
            (0xFFC00000, QNAN), (0x7F7FFFFF, 0x43000000)]   # FLT_MAX -> 128 - 2^-23, nearest float32 is 128
    got = bits(palog2(f32([r[0] for r in rows])))
    bad = [(hex(r[0]), hex(int(g)), hex(r[1])) for r, g in zip(rows, got) if int(g) != r[1]]
    assert not bad, f"palog2 special cases differ: {bad}"


PALOG2_CHECKS = [check_palog2_golden, check_palog2_powers_and_first_octaves, check_palog2_nearest,
                 check_palog2_mitchell_bounds, check_palog2_monotone, check_palog2_specials]


# ---------------------------------------------------------------------------
# paexp2
# ---------------------------------------------------------------------------

def check_paexp2_golden(paexp2):
    cases = load_golden("paexp2")
    got = bits(paexp2(f32([c[0] for c in cases])))
    bad = [c[3] for c, g in zip(cases, got) if int(g) != c[2]]
    assert not bad, f"paexp2 golden cases differ: {bad}"


def check_paexp2_integers_and_exact(paexp2):
    """paexp2(k) = 2^k; for |A| >= 1 the fraction has at most 23 bits, so
    2^floor(A) (1 + frac) is exact."""
    k = np.arange(-126, 128)
    got = paexp2(k.astype(np.float32))
    assert np.array_equal(bits(got), bits(np.ldexp(np.float32(1.0), k).astype(np.float32)))
    g = np.random.default_rng(31)
    x = (g.uniform(-126, 128, size=20000)).astype(np.float32)
    x = x[np.abs(x) >= 1.0]
    got = bits(paexp2(x))
    for xv, z in zip(x[:3000], got[:3000]):
        q = Fraction(float(xv))
        fl = math.floor(q)
        want = Fraction(2) ** fl * (1 + q - fl)
        assert exact(int(z)) == want, (float(xv), hex(z))


def check_paexp2_nearest(paexp2):
    """For |A| < 1 the exact value needs rounding: nearest float32, ties to even
    (R14), including constructed ties."""
    g = np.random.default_rng(32)
    e = g.integers(-40, 0, size=2000)
    m = g.integers(0, 1 << 23, size=2000)
    s = g.integers(0, 2, size=2000)
    x = ((s << 31) | ((e + 127) << 23) | m).astype(np.uint32).view(np.float32)
    ties = f32([0x33800000, 0x34400000, 0xB3000000, 0xB3400000, 0x33C00000, 0x34200000])  # 2^-24, 3*2^-24, ...
    x = np.concatenate([x, ties])
    got = bits(paexp2(x))
    for xv, z in zip(x, got):
        q = Fraction(float(xv))
        fl = math.floor(q)
        want = Fraction(2) ** fl * (1 + q - fl)
        assert is_nearest_even(int(z), want), (float(xv), hex(z))


def check_paexp2_bounds(paexp2):
    """2^A <= paexp2(A) <= 1.0615 * 2^A (1 + f >= 2^f on [0, 1))."""
    x = np.random.default_rng(33).uniform(-120, 120, size=20000).astype(np.float32)
    got = paexp2(x).astype(np.float64)
    ref = np.exp2(x.astype(np.float64))
    assert np.all(got >= ref * (1 - 2.0 ** -23))
    assert np.all(got <= ref * 1.06154 * (1 + 2.0 ** -23))


def check_paexp2_inverts_palog2(paexp2):
    """paexp2(palog2(x)) = x where palog2 is exact (x in [1/2, 2))."""
    m = np.random.default_rng(34).integers(0, 1 << 23, size=20000)
    for hi in (0x3F800000, 0x3F000000):
        x = (hi | m).astype(np.uint32).view(np.float32)
        lg = (m / float(1 << 23) - (0.0 if hi == 0x3F800000 else 1.0)).astype(np.float32)   # E + M, exact
        assert np.array_equal(bits(paexp2(lg)), bits(x))


def check_paexp2_monotone(paexp2):
    x = np.sort(np.random.default_rng(35).uniform(-130, 130, size=50000).astype(np.float32))
    got = paexp2(x).astype(np.float64)
    assert np.all(got[1:] >= got[:-1])


def check_paexp2_specials(paexp2):
    """Reading R14 (parity pinned by reading)."""
    rows = [(0x7F800000, 0x7F800000), (0xFF800000, 0x00000000), (0x7FC00000, QNAN), (0xFFC00123, QNAN),
            (0x43000000, 0x7F800000),            # 128 -> 2^128 overflows
            (0x42FFFFFF, 0x7F7FFFC0),            # 128 - 2^-17 -> 2^127 (2 - 2^-17), exact
            (0xC2FC0000, 0x00800000),            # -126 -> 2^-126
            (0xC2FE0000, 0x00000000),            # -127 -> below min normal -> +0
            (0x00000003, 0x3F800000), (0x80000003, 0x3F800000), (0x80000000, 0x3F800000)]
    got = bits(paexp2(f32([r[0] for r in rows])))
    bad = [(hex(r[0]), hex(int(g)), hex(r[1])) for r, g in zip(rows, got) if int(g) != r[1]]
    assert not bad, f"paexp2 special cases differ: {bad}"


PAEXP2_CHECKS = [check_paexp2_golden, check_paexp2_integers_and_exact, check_paexp2_nearest, check_paexp2_bounds,
                 check_paexp2_inverts_palog2, check_paexp2_monotone, check_paexp2_specials]
