"""CPU oracle for the other elementwise piecewise affine operations.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the HIP library and never calls it.

Source: Kosson & Jaggi, "Multiplication-Free Transformer Training via
Piecewise Affine Operations" (NeurIPS 2023), Sec. 2.3 (Other Piecewise Affine
Operations):

  * paexp2(A) = 2^floor(A) (1 + A - floor(A)),
  * palog2(A) = E_A + M_A for A = 2^E_A (1 + M_A) > 0,
  * piecewise affine division A ./ B (PAD), the inverse of PAM, with sign
    S_A - S_B, exponent E_A - E_B - borrow and mantissa M_A - M_B + borrow;
    for float32 it is the int32 difference of the two encodings plus one
    exponent bias (127 << 23); for positive numbers it equals
    paexp2(palog2 A - palog2 B).

Readings where the paper is silent, loose or garbled (hard-coded here and in
the HIP library):

  R10 PAD borrow.  The printed exponent line subtracts 1{M_A - M_B <= 0} and
      the printed mantissa line adds 1{M_A - M_B <= 1}; taken literally the
      mantissa leaves [0, 1) whenever M_A > M_B.  Read as the borrow of the
      int32 subtraction the same passage describes: 1{M_A - M_B < 0} in both
      lines.
  R12 PAD edge cases, in the spirit of R1-R6 for PAM: sign = S_A - S_B taken
      mod 2 (exclusive or); denormal operands count as zero; a NaN operand,
      0 ./ 0 and inf ./ inf give the canonical NaN 0x7FC00000; x ./ 0 and
      inf ./ x give a signed inf (x nonzero finite, or inf over zero);
      0 ./ x and x ./ inf give a signed zero; a result whose exponent field
      would be <= 0 is a signed zero, >= 255 is +-FLT_MAX.
  R13 palog2 returns float32: the real value E_A + M_A rounded to the nearest
      float32 (ties to even).  Outside A > 0 it follows log2: +-0 and
      denormals give -inf, negative A gives NaN, +inf gives +inf, NaN gives
      NaN (always 0x7FC00000).
  R14 paexp2 returns float32: the real value 2^floor(A) (1 + A - floor(A))
      rounded to the nearest float32 (ties to even).  Results below 2^-126
      are +0 (denormals flushed, as R4); results above FLT_MAX are +inf (as
      exp2); -inf gives +0, +inf gives +inf, NaN gives 0x7FC00000.

Two renderings are given for PAD (bit form and field form) and for palog2 /
paexp2 (integer form and exact-rational form); the tests check them against
each other and against closed forms the paper fixes.
"""
from __future__ import annotations

from fractions import Fraction
import math

import numpy as np

SIGN = 0x80000000
MAG = 0x7FFFFFFF
BIAS = 127 << 23           # 0x3F800000
MIN_NORMAL = 0x00800000
FLT_MAX = 0x7F7FFFFF
INF = 0x7F800000
NEG_INF = 0xFF800000
QNAN = 0x7FC00000


# ---------------------------------------------------------------------------
# PAD, scalar forms
# ---------------------------------------------------------------------------

def pad_bits(ua: int, ub: int) -> int:
    """Bit form: the int32 difference of the encodings plus one bias (Sec. 2.3)."""
    s = (ua ^ ub) & SIGN                       # R12: S_A - S_B mod 2
    ma = ua & MAG
    mb = ub & MAG
    if ma > INF or mb > INF:
        return QNAN
    a_zero = ma < MIN_NORMAL
    b_zero = mb < MIN_NORMAL
    if ma == INF:
        return QNAN if mb == INF else s | INF
    if mb == INF:
        return s                               # finite ./ inf
    if a_zero:
        return QNAN if b_zero else s           # 0 ./ 0, 0 ./ x
    if b_zero:
        return s | INF                         # x ./ 0
    t = ma - mb + BIAS                         # subtract encodings, restore one bias
    if t < MIN_NORMAL:
        return s
    if t > FLT_MAX:
        return s | FLT_MAX
    return s | t


def pad_fields(ua: int, ub: int) -> int:
    """Field form: Sec. 2.3's sign / exponent / mantissa lines with R10's borrow.

    Shares no arithmetic with ``pad_bits``.
    """
    sa, ea, fa = ua >> 31, (ua >> 23) & 0xFF, ua & 0x7FFFFF
    sb, eb, fb = ub >> 31, (ub >> 23) & 0xFF, ub & 0x7FFFFF
    s = (sa - sb) % 2
    if (ea == 255 and fa) or (eb == 255 and fb):
        return QNAN
    a_inf, b_inf = ea == 255, eb == 255
    a_zero, b_zero = ea == 0, eb == 0
    if a_inf and b_inf:
        return QNAN
    if a_inf:
        return (s << 31) | (255 << 23)
    if b_inf:
        return s << 31
    if a_zero and b_zero:
        return QNAN
    if a_zero:
        return s << 31
    if b_zero:
        return (s << 31) | (255 << 23)
    borrow = 1 if fa - fb < 0 else 0           # 1{M_A - M_B < 0}  (R10)
    e = (ea - 127) - (eb - 127) - borrow
    f = fa - fb + borrow * (1 << 23)
    if e < -126:
        return s << 31
    if e > 127:
        return (s << 31) | FLT_MAX
    return (s << 31) | ((e + 127) << 23) | f


# ---------------------------------------------------------------------------
# palog2 / paexp2, exact-rational forms (scalar)
# ---------------------------------------------------------------------------

def round_to_f32_bits(q: Fraction) -> int:
    """Nearest float32 to a positive rational q (ties to even), as bits.

    Written out with exact rationals: find E with 2^E <= q < 2^(E+1), round
    q / 2^E * 2^23 to an integer (ties to even), renormalise a carry, then
    flush below 2^-126 to +0 and send above FLT_MAX to +inf.
    """
    assert q > 0
    e = q.numerator.bit_length() - q.denominator.bit_length()
    if Fraction(2) ** e > q:
        e -= 1
    while Fraction(2) ** (e + 1) <= q:
        e += 1
    scaled = q / Fraction(2) ** e * (1 << 23)          # in [2^23, 2^24)
    n = math.floor(scaled)
    rem = scaled - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    if n == 1 << 24:
        n >>= 1
        e += 1
    if e < -126:
        return 0
    if e > 127:
        return INF
    return ((e + 127) << 23) | (n - (1 << 23))


def f32_value(u: int) -> Fraction:
    """Exact value of a finite float32 encoding (denormals included)."""
    s, ex, fr = u >> 31, (u >> 23) & 0xFF, u & 0x7FFFFF
    if ex == 0:
        v = Fraction(fr, 1 << 23) * Fraction(2) ** -126
    else:
        v = (1 + Fraction(fr, 1 << 23)) * Fraction(2) ** (ex - 127)
    return -v if s else v


def palog2_exact(u: int) -> int:
    """palog2 of one float32 encoding via exact rationals (R13)."""
    s, ex, fr = u >> 31, (u >> 23) & 0xFF, u & 0x7FFFFF
    if ex == 255:
        return QNAN if (fr or s) else INF
    if ex == 0:
        return NEG_INF                         # +-0 and denormals (DAZ)
    if s:
        return QNAN
    v = Fraction(ex - 127) + Fraction(fr, 1 << 23)   # E_A + M_A
    if v == 0:
        return 0
    mag = round_to_f32_bits(abs(v))
    return mag | (SIGN if v < 0 else 0)


def paexp2_exact(u: int) -> int:
    """paexp2 of one float32 encoding via exact rationals (R14)."""
    s, ex, fr = u >> 31, (u >> 23) & 0xFF, u & 0x7FFFFF
    if ex == 255:
        if fr:
            return QNAN
        return 0 if s else INF
    a = f32_value(u) if ex != 0 else Fraction(0)     # denormal input counts as zero
    fl = math.floor(a)
    if fl > 200:
        return INF
    if fl < -200:
        return 0
    q = Fraction(2) ** fl * (1 + a - fl)
    return round_to_f32_bits(q)


# ---------------------------------------------------------------------------
# Vectorised forms (numpy)
# ---------------------------------------------------------------------------

def _u(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.int64)


def _f(u: np.ndarray) -> np.ndarray:
    return np.asarray(u).astype(np.uint32).view(np.float32)


def pad_ref(a, b) -> np.ndarray:
    """Elementwise PAD of float32 arrays (broadcasting), bit form."""
    a = np.asarray(a, dtype=np.float32)
    b = np.asarray(b, dtype=np.float32)
    a, b = np.broadcast_arrays(a, b)
    ua, ub = _u(a), _u(b)
    s = (ua ^ ub) & SIGN
    ma, mb = ua & MAG, ub & MAG
    t = ma - mb + BIAS
    out = np.where(t > FLT_MAX, s | FLT_MAX, s | t)
    out = np.where(t < MIN_NORMAL, s, out)
    a_zero, b_zero = ma < MIN_NORMAL, mb < MIN_NORMAL
    out = np.where(b_zero, s | INF, out)                      # x ./ 0
    out = np.where(a_zero, np.where(b_zero, QNAN, s), out)    # 0 ./ x, 0 ./ 0
    out = np.where(mb == INF, s, out)                         # x ./ inf
    out = np.where(ma == INF, np.where(mb == INF, QNAN, s | INF), out)
    out = np.where((ma > INF) | (mb > INF), QNAN, out)
    return _f(out)


def palog2_ref(a) -> np.ndarray:
    """Elementwise palog2 of a float32 array (R13)."""
    a = np.asarray(a, dtype=np.float32)
    u = _u(a)
    mag = u & MAG
    # E_A + M_A = (encoding - 127 * 2^23) / 2^23: exact in float64, then one
    # rounding to float32 (ties to even).
    val = ((mag - BIAS).astype(np.float64) / float(1 << 23)).astype(np.float32)
    out = val.view(np.uint32).astype(np.int64)
    out = np.where(mag < MIN_NORMAL, NEG_INF, out)
    out = np.where((u >= SIGN) & (mag >= MIN_NORMAL), QNAN, out)
    out = np.where(u == INF, INF, out)
    out = np.where(mag > INF, QNAN, out)
    return _f(out)


def paexp2_ref(a) -> np.ndarray:
    """Elementwise paexp2 of a float32 array (R14).

    2^floor(A) (1 + A - floor(A)) has the float32 encoding A * 2^23 + 127 *
    2^23 read as a fixed-point number; rounding A * 2^23 to the nearest
    integer (ties to even) rounds the result to the nearest float32, a carry
    out of the mantissa moving into the exponent as it should.
    """
    a = np.asarray(a, dtype=np.float32)
    u = _u(a)
    mag = u & MAG
    x = np.where((mag < MIN_NORMAL) | (mag > INF), np.float32(0.0), a).astype(np.float64)  # denormals count as zero
    x = np.clip(np.nan_to_num(x, posinf=256.0, neginf=-256.0), -256.0, 256.0)
    r = np.rint(x * float(1 << 23)).astype(np.int64)       # exact product, ties to even
    enc = r + BIAS
    out = np.where(enc >= INF, INF, enc)
    out = np.where(enc < MIN_NORMAL, 0, out)
    out = np.where(mag > INF, QNAN, out)
    return _f(out)
