"""CPU oracle for piecewise affine multiplication (PAM) and PAM matrix products.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the HIP library and never calls it.

Source: Kosson & Jaggi, "Multiplication-Free Transformer Training via
Piecewise Affine Operations" (NeurIPS 2023).

  * Sec. 2.1 (Floating Point Numbers): a float32 is [S, E-bar (8 bits, bias
    127), M-bar (23 bits)], value (-1)^S 2^E (1 + M) with E = E-bar - 127 and
    M = M-bar / 2^23; E-bar = 255 encodes inf/NaN, E-bar = 0 zero/denormals.
  * Sec. 2.2 (Piecewise Affine Multiplication): A .^ B has sign S_A + S_B,
    exponent E_A + E_B + 1{M_A + M_B >= 1} and mantissa
    M_A + M_B - 1{M_A + M_B >= 1}.  For float32 this is the int32 sum of the
    two bit patterns minus one exponent bias (127 << 23), with exponent
    under/overflow clamped, denormals flushed and NaN/inf handled explicitly.
  * Sec. 2.3 (Other Piecewise Affine Operations): the same product is
    paexp2(palog2 A + palog2 B) for positive A, B.
  * Sec. 3.2 (Replacing Matrix Multiplications) and Table 1: a PAM matrix
    product replaces every scalar product of a matrix multiply by PAM and
    keeps ordinary addition; the backward products (approximate derivative)
    are the same kind of product with transposed operands.
  * App. "Hardware Cost" and App. "PAM with Narrower Mantissas": accumulation
    stays ordinary floating-point addition.

Readings where the paper is silent or loose (each one is hard-coded here and
in the HIP library):

  R1  sign = S_A + S_B taken mod 2 (exclusive or); a zero result carries it.
  R2  a zero operand gives a signed zero.
  R3  denormal operands count as zero (the paper allows flushing them).
  R4  underflow (result exponent field <= 0) gives a signed zero; clamping the
      exponent field to 0 leaves a denormal encoding, which is flushed.
  R5  overflow (result exponent field >= 255) saturates to +-FLT_MAX, the
      largest finite value (the paper clamps overflowing results to the
      maximum), which keeps |A .^ B| <= |A * B| for all finite operands.
  R6  NaN operand -> NaN; inf times zero/denormal -> NaN; inf times anything
      else -> signed inf.  NaN results are the canonical quiet NaN 0x7FC00000.
  R7  the bias removed is 127 << 23 = 0x3F800000, once, from the magnitude
      sum; the mantissa carry into the exponent realises 1{M_A + M_B >= 1}.
  R8  matrix products accumulate in floating point in an unspecified order;
      this oracle accumulates in float64 in increasing k, and also returns
      S = sum_k |term| so that callers can bound float32 rounding.

  R11 narrower mantissas (App. "PAM with Narrower Mantissas": inputs are
      rounded and their extra mantissa bits masked, accumulation unchanged):
      each input is rounded to the nearest float32 whose mantissa has m
      significant bits (ties to even), a carry moving into the exponent and
      a finite value rounding past FLT_MAX becoming inf, as a narrower
      float format's conversion does; inf stays inf and NaN stays NaN.  The
      rounded inputs then go through PAM (R1-R7) with float32 accumulation.

  R15 exact derivative (Table 1: d(A .^ B)/dA = 2^(E_B + 1{M_A + M_B >= 1})
      with no sign and no edge cases; Sec. "Derivatives": the exact
      derivative is the true, piecewise constant derivative of the piecewise
      affine function):
      * the sign of B is part of it: d(A .^ B)/dA = sgn(B) 2^(E_B + c) for
        either sign of A, since the magnitude of A .^ B grows with |A| and its
        sign is S_A + S_B;
      * it is 0 wherever A .^ B is clamped to a constant: a zero or denormal A
        or B (R2, R3), a result that underflows to a signed zero (R4: the
        magnitude sum |A| + |B| - bias below 0x00800000) and a result that
        saturates at +-FLT_MAX (R5: that sum above 0x7F7FFFFF) -- the function
        is flat there, so its true derivative is zero;
      * elsewhere (the sum in [0x00800000, 0x7F7FFFFF], the result not
        clamped) it is Table 1's power of two.  That is the slope of the
        affine piece A .^ B follows as |A| grows from A (where the carry
        flips, 1{M_A + M_B >= 1} takes the upper piece); at a sum of exactly
        0x7F7FFFFF, the unclamped FLT_MAX itself, the slope of the piece below
        (e.g. d(A .^ 1)/dA = 1 for every normal A, FLT_MAX included).
      For a matrix product Y = X .^ W^T the exact derivatives are
        dX[i,k] = sum_j dY[i,j] d(X[i,k] .^ W[j,k])/dX[i,k]
        dW[j,k] = sum_i dY[i,j] d(W[j,k] .^ X[i,k])/dW[j,k].
      Each term dY * g with g a power of two is exact (Sec. "Derivatives":
      such a product is performed exactly by PAM), and PAM reads a denormal
      operand as zero (R3), so a denormal dY contributes nothing; the terms
      are accumulated in float32 (here: float64, plus S = sum |terms|).
      A term whose exact value leaves the float32 range is kept exact here;
      the float32 sum rounds it like any other addend.  Inf / NaN operands
      are outside this reading (parity unpinned there).

Three independent renderings of the scalar product are given (bit, field and
value form); the tests check them against each other and against the facts
the paper states.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence, Tuple

import numpy as np

SIGN = 0x80000000
MAG = 0x7FFFFFFF
BIAS = 127 << 23           # 0x3F800000, the float32 encoding of 1.0
MIN_NORMAL = 0x00800000    # 2^-126
FLT_MAX = 0x7F7FFFFF
INF = 0x7F800000
QNAN = 0x7FC00000


# ---------------------------------------------------------------------------
# Scalar forms
# ---------------------------------------------------------------------------

def pam_bits(ua: int, ub: int) -> int:
    """Bit form: Sec. 2.2, the int32 addition of the two float32 encodings.

    ua, ub are float32 bit patterns (Python ints in [0, 2^32)).
    """
    s = (ua ^ ub) & SIGN                       # R1
    ma = ua & MAG
    mb = ub & MAG
    if ma > INF or mb > INF:                   # R6: NaN operand
        return QNAN
    if ma == INF or mb == INF:                 # R6: an infinite operand
        other = mb if ma == INF else ma
        if other < MIN_NORMAL:
            return QNAN
        return s | INF
    if ma < MIN_NORMAL or mb < MIN_NORMAL:     # R2, R3
        return s
    t = ma + mb - BIAS                         # add encodings, drop one bias (R7)
    if t < MIN_NORMAL:                         # R4
        return s
    if t > FLT_MAX:                            # R5
        return s | FLT_MAX
    return s | t


def pam_fields(ua: int, ub: int) -> int:
    """Field form: Sec. 2.2, sign/exponent/mantissa definition applied literally.

    Decodes (S, E, M-bar) of each operand, forms the carry 1{M_A + M_B >= 1},
    the exponent E_A + E_B + carry and the mantissa M_A + M_B - carry, then
    re-encodes.  Shares no arithmetic with ``pam_bits``.
    """
    sa, ea, fa = ua >> 31, (ua >> 23) & 0xFF, ua & 0x7FFFFF
    sb, eb, fb = ub >> 31, (ub >> 23) & 0xFF, ub & 0x7FFFFF
    s = (sa + sb) % 2                          # R1
    a_nan = ea == 255 and fa != 0
    b_nan = eb == 255 and fb != 0
    a_inf = ea == 255 and fa == 0
    b_inf = eb == 255 and fb == 0
    if a_nan or b_nan:
        return QNAN
    if a_inf or b_inf:
        other_zero = (eb == 0) if a_inf else (ea == 0)
        if other_zero:
            return QNAN
        return (s << 31) | (255 << 23)
    if ea == 0 or eb == 0:                     # zero or denormal operand
        return s << 31
    e_a = ea - 127
    e_b = eb - 127
    carry = 1 if fa + fb >= (1 << 23) else 0   # 1{M_A + M_B >= 1}
    e = e_a + e_b + carry
    f = fa + fb - carry * (1 << 23)
    if e < -126:                               # R4
        return s << 31
    if e > 127:                                # R5
        return (s << 31) | FLT_MAX
    return (s << 31) | ((e + 127) << 23) | f


def palog2(x: float) -> float:
    """Sec. 2.3: palog2(A) = E_A + M_A for A > 0 (A = 2^E (1 + M))."""
    m, e = math.frexp(x)                       # x = m 2^e, m in [0.5, 1)
    return (e - 1) + (2.0 * m - 1.0)


def paexp2(x: float) -> float:
    """Sec. 2.3: paexp2(A) = 2^floor(A) (1 + A - floor(A))."""
    fl = math.floor(x)
    return math.ldexp(1.0 + (x - fl), fl)


def pam_value(a: float, b: float) -> float:
    """Value form: Sec. 2.3, paexp2(palog2|A| + palog2|B|) with the sign of A*B.

    Exact in float64 for float32 inputs (palog2 needs at most 8 + 23 bits).
    Only for finite normal operands; returns the unclamped real value, or
    0.0 / FLT_MAX after R4 / R5.
    """
    mag = paexp2(palog2(abs(a)) + palog2(abs(b)))
    neg = (math.copysign(1.0, a) < 0) != (math.copysign(1.0, b) < 0)
    if mag < 2.0 ** -126:
        mag = 0.0
    elif mag > float(np.finfo(np.float32).max):
        mag = float(np.finfo(np.float32).max)
    return -mag if neg else mag


# ---------------------------------------------------------------------------
# Vectorised bit form (numpy), same steps as ``pam_bits``
# ---------------------------------------------------------------------------

def pam_mul_ref(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Elementwise PAM of float32 arrays (broadcasting), bit form of Sec. 2.2."""
    a = np.asarray(a, dtype=np.float32)
    b = np.asarray(b, dtype=np.float32)
    ua = a.view(np.uint32).astype(np.int64)
    ub = b.view(np.uint32).astype(np.int64)
    s = (ua ^ ub) & SIGN
    ma = ua & MAG
    mb = ub & MAG
    t = ma + mb - BIAS
    out = np.where(t > FLT_MAX, s | FLT_MAX, s | t)           # R5
    out = np.where(t < MIN_NORMAL, s, out)                    # R4
    out = np.where((ma < MIN_NORMAL) | (mb < MIN_NORMAL), s, out)  # R2, R3
    a_inf = ma == INF
    b_inf = mb == INF
    inf_res = np.where((a_inf & (mb < MIN_NORMAL)) | (b_inf & (ma < MIN_NORMAL)), QNAN, s | INF)
    out = np.where(a_inf | b_inf, inf_res, out)               # R6
    out = np.where((ma > INF) | (mb > INF), QNAN, out)        # R6
    return out.astype(np.uint32).view(np.float32)


# ---------------------------------------------------------------------------
# Narrower mantissas (R11)
# ---------------------------------------------------------------------------

def round_mantissa_bits(u: int, bits: int) -> int:
    """One float32 encoding rounded to ``bits`` mantissa bits (R11), scalar form.

    Works on the value: decode, round the significand 1.M (or 0.M for a
    denormal) to a multiple of 2^-bits with ties to even, re-encode.
    """
    s, ex, fr = u >> 31, (u >> 23) & 0xFF, u & 0x7FFFFF
    if ex == 255:
        return u
    drop = 23 - bits
    if drop == 0:
        return u
    sig = fr | ((1 << 23) if ex else 0)            # 24-bit significand (23 for denormals)
    q, r = divmod(sig, 1 << drop)
    half = 1 << (drop - 1)
    if r > half or (r == half and (q & 1)):
        q += 1
    sig = q << drop
    e = ex if ex else 1
    if sig >= (1 << 24):                            # carry out of the significand
        sig >>= 1
        e += 1
    if ex == 0 and sig >= (1 << 23):                # a denormal rounded up to the min normal
        e, sig = 1, sig
        return (s << 31) | (1 << 23) | (sig - (1 << 23))
    if ex == 0:
        return (s << 31) | sig
    if e >= 255:
        return (s << 31) | INF
    return (s << 31) | (e << 23) | (sig - (1 << 23))


def round_mantissa_scalar_ref(x: np.ndarray, bits: int) -> np.ndarray:
    """Elementwise R11 rounding through the scalar value form (slow)."""
    x = np.asarray(x, dtype=np.float32)
    u = x.view(np.uint32).reshape(-1)
    out = np.fromiter((round_mantissa_bits(int(v), bits) for v in u), dtype=np.uint32, count=u.size)
    return out.view(np.float32).reshape(x.shape)


def round_mantissa_ref(x: np.ndarray, bits: int) -> np.ndarray:
    """Elementwise R11 rounding of a float32 array to ``bits`` mantissa bits.

    On the encoding: the dropped low bits decide the rounding (above half, or
    exactly half with an odd kept part, rounds the kept part up); a carry out
    of the mantissa moves into the exponent, and past the largest exponent
    lands on the inf encoding.  inf and NaN encodings are left as they are.
    """
    if not 0 <= bits <= 23:
        raise ValueError("bits must be in [0, 23]")
    x = np.asarray(x, dtype=np.float32)
    if bits == 23:
        return x.copy()
    u = x.view(np.uint32).astype(np.int64)
    drop = 23 - bits
    low = u & ((1 << drop) - 1)
    kept = u >> drop
    half = 1 << (drop - 1)
    up = (low > half) | ((low == half) & ((kept & 1) == 1))
    r = (kept + up.astype(np.int64)) << drop                 # may carry into the exponent (and up to inf)
    r = np.where((u & INF) == INF, u, r)
    return r.astype(np.uint32).view(np.float32)


# ---------------------------------------------------------------------------
# PAM matrix product
# ---------------------------------------------------------------------------

def op(x: np.ndarray, trans: bool) -> np.ndarray:
    """op(X) = X^T when trans else X (row-major storage, Sec. 3.2 forms)."""
    return x.T if trans else x


def pam_gemm_ref(a: np.ndarray, b: np.ndarray, trans_a: bool = False, trans_b: bool = False,
                 rows: Optional[Sequence[int]] = None,
                 cols: Optional[Sequence[int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """C[i, j] = sum_k pam(op(A)[i, k], op(B)[k, j]) (Sec. 3.2).

    Returns (C, S) in float64, where S[i, j] = sum_k |pam(...)|.  ``rows`` and
    ``cols`` restrict the output to a sub-grid (for sampled checks of large
    products).  Accumulation is float64 in increasing k.
    """
    opa = op(np.asarray(a, dtype=np.float32), trans_a)
    opb = op(np.asarray(b, dtype=np.float32), trans_b)
    m, k = opa.shape
    k2, n = opb.shape
    if k != k2:
        raise ValueError("inner dimensions differ")
    if rows is not None:
        opa = opa[np.asarray(rows, dtype=np.int64), :]
    if cols is not None:
        opb = opb[:, np.asarray(cols, dtype=np.int64)]
    c = np.zeros((opa.shape[0], opb.shape[1]), dtype=np.float64)
    s = np.zeros_like(c)
    # inf terms of opposite signs make a NaN sum, as IEEE addition defines;
    # numpy's warning about it carries no information here
    with np.errstate(invalid="ignore"):
        for kk in range(k):
            term = pam_mul_ref(opa[:, kk:kk + 1], opb[kk:kk + 1, :]).astype(np.float64)
            c += term
            s += np.abs(term)
    return c, s


def pam_gemm_batched_ref(a: np.ndarray, b: np.ndarray, trans_a: bool = False, trans_b: bool = False,
                         batches: Optional[Sequence[int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Independent PAM products over the leading batch axis (Sec. 3.2, attention)."""
    idx = range(a.shape[0]) if batches is None else batches
    cs, ss = [], []
    for i in idx:
        c, s = pam_gemm_ref(a[i], b[i], trans_a, trans_b)
        cs.append(c)
        ss.append(s)
    return np.stack(cs), np.stack(ss)


def pam_exact_grad_factor(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """d(a .^ b)/da in float64 (Table 1, reading R15), elementwise, broadcasting.

    sgn(b) 2^(E_b + 1{M_a + M_b >= 1}) where a .^ b is not clamped, 0 where it
    is (zero / denormal operand, underflow, saturation).  Finite operands only.
    """
    a = np.asarray(a, dtype=np.float32)
    b = np.asarray(b, dtype=np.float32)
    ua = a.view(np.uint32).astype(np.int64)
    ub = b.view(np.uint32).astype(np.int64)
    ea, eb = (ua >> 23) & 0xFF, (ub >> 23) & 0xFF
    fa, fb = ua & 0x7FFFFF, ub & 0x7FFFFF
    carry = ((fa + fb) >= (1 << 23)).astype(np.int64)          # 1{M_A + M_B >= 1}
    sign = np.where(ub >> 31 == 1, -1.0, 1.0)
    g = sign * np.ldexp(1.0, (eb - 127 + carry).astype(np.int64))
    t = (ua & MAG) + (ub & MAG) - BIAS                         # magnitude of a .^ b before R4 / R5
    flat = (ea == 0) | (eb == 0) | (t < MIN_NORMAL) | (t > FLT_MAX)
    return np.where(flat, 0.0, g)


def pam_exact_grads_ref(dy: np.ndarray, x: np.ndarray, w: np.ndarray):
    """Exact derivatives of Y = X .^ W^T (Table 1, R15): (dX, S_dX, dW, S_dW)
    in float64, S = sum of |terms|.  dy [T, N], x [T, K], w [N, K]."""
    dy = np.asarray(dy, dtype=np.float32)
    # a denormal dY is a zero operand of the term's PAM (R3)
    dy = np.where(np.abs(dy) < np.float32(2.0 ** -126), np.float32(0.0), dy).astype(np.float64)
    t, n = dy.shape
    k = np.asarray(x).shape[1]
    dx = np.zeros((t, k))
    sdx = np.zeros((t, k))
    dw = np.zeros((n, k))
    sdw = np.zeros((n, k))
    for j in range(n):
        gx = pam_exact_grad_factor(x, w[j:j + 1, :])                  # [T, K]: d(X .^ W[j])/dX
        term = dy[:, j:j + 1] * gx
        dx += term
        sdx += np.abs(term)
        gw = pam_exact_grad_factor(w[j:j + 1, :], x)                  # [T, K]: d(W[j] .^ X)/dW[j]
        term = dy[:, j:j + 1] * gw
        dw[j] = term.sum(axis=0)
        sdw[j] = np.abs(term).sum(axis=0)
    return dx, sdx, dw, sdw


def gemm_tolerance(s: np.ndarray, k: int) -> np.ndarray:
    """Allowed |C_fp32 - C_ref|: 1e-5 * sqrt(K) relative to sum_k |term|.

    Plus K * 2^-126 for partial sums flushed to zero as denormals.
    """
    return 1e-5 * math.sqrt(max(k, 1)) * s + max(k, 1) * 2.0 ** -126
