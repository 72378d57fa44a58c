"""Planted mistakes in copies of the oracle must be caught by the pins.

Each mutant is a plausible slip (a dropped term, a wrong constant, sign or
index, a transposed operand).  The test passes only if at least one pin
rejects every mutant, which shows that the pins constrain the oracle rather
than restate it.  Mutants live here, on the CPU; the oracle itself is not
modified.
"""
import numpy as np
import pytest

import pins
from oracle import pam_ref

SIGN, MAG, BIAS = 0x80000000, 0x7FFFFFFF, 0x3F800000
MIN_NORMAL, FLT_MAX, INF, QNAN = 0x00800000, 0x7F7FFFFF, 0x7F800000, 0x7FC00000


def vec(fn):
    def mul(a, b):
        a = np.asarray(a, dtype=np.float32)
        b = np.asarray(b, dtype=np.float32)
        a, b = np.broadcast_arrays(a, b)
        ua = a.view(np.uint32).reshape(-1)
        ub = b.view(np.uint32).reshape(-1)
        out = np.fromiter((fn(int(x), int(y)) for x, y in zip(ua, ub)), dtype=np.uint32, count=ua.size)
        return out.view(np.float32).reshape(a.shape)
    return mul


def make_scalar(bias=BIAS, sign_op="xor", under="lt", over="flt_max", flush_denormal=True,
                drop_mag_b=False, nan_inf=True):
    def f(ua, ub):
        s = ((ua ^ ub) if sign_op == "xor" else (ua | ub)) & SIGN
        ma, mb = ua & MAG, ub & MAG
        if nan_inf:
            if ma > INF or mb > INF:
                return QNAN
            if ma == INF or mb == INF:
                other = mb if ma == INF else ma
                return QNAN if other < MIN_NORMAL else s | INF
        if flush_denormal and (ma < MIN_NORMAL or mb < MIN_NORMAL):
            return s
        t = ma + (0 if drop_mag_b else mb) - bias
        if (t < MIN_NORMAL) if under == "lt" else (t <= MIN_NORMAL):
            return s
        if t > FLT_MAX:
            return s | (FLT_MAX if over == "flt_max" else INF)
        return s | (t & MAG)
    return f


SCALAR_MUTANTS = {
    "no_bias": make_scalar(bias=0),
    "bias_wrong_shift": make_scalar(bias=127 << 22),
    "bias_off_by_one_exponent": make_scalar(bias=126 << 23),
    "sign_or": make_scalar(sign_op="or"),
    "underflow_off_by_one": make_scalar(under="le"),
    "overflow_to_inf": make_scalar(over="inf"),
    "denormals_not_flushed": make_scalar(flush_denormal=False),
    "dropped_operand": make_scalar(drop_mag_b=True),
}


def caught(checks, *args):
    for check in checks:
        try:
            check(*args)
        except AssertionError:
            return check.__name__
    return None


def test_unmutated_oracle_passes_scalar_pins():
    assert caught(pins.SCALAR_CHECKS[:3] + [pins.check_range_readings], vec(pam_ref.pam_bits)) is None


@pytest.mark.parametrize("name", sorted(SCALAR_MUTANTS))
def test_scalar_mutant_is_caught(name):
    mul = vec(SCALAR_MUTANTS[name])
    cheap = [pins.check_golden, pins.check_max_error_example, pins.check_range_readings,
             pins.check_error_bounds, pins.check_value_form]
    assert caught(cheap, mul) is not None, f"mutant {name} passed every pin"


def field_no_carry(ua, ub):
    """Field form with the carry into the exponent dropped (mantissa wraps)."""
    ea, fa = (ua >> 23) & 0xFF, ua & 0x7FFFFF
    eb, fb = (ub >> 23) & 0xFF, ub & 0x7FFFFF
    s = ((ua >> 31) + (ub >> 31)) % 2
    if ea == 0 or eb == 0 or ea == 255 or eb == 255:
        return pam_ref.pam_fields(ua, ub)
    e = (ea - 127) + (eb - 127)
    f = (fa + fb) & 0x7FFFFF
    if e < -126:
        return s << 31
    if e > 127:
        return (s << 31) | FLT_MAX
    return (s << 31) | ((e + 127) << 23) | f


def test_field_form_mutant_is_caught():
    assert caught([pins.check_golden, pins.check_error_bounds], vec(field_no_carry)) is not None


def gemm_mutant(kind):
    def gemm(a, b, ta, tb):
        if kind == "square_b_read_untransposed":
            # reads B[k*ldb + j] instead of B[j*ldb + k]; only shape-consistent for square B
            if tb and b.shape[0] == b.shape[1]:
                tb = False
        if kind == "swap_trans" and (a.T if tb else a).shape[1] == (b.T if ta else b).shape[0]:
            ta, tb = tb, ta
        c, s = pam_ref.pam_gemm_ref(a, b, ta, tb)
        if kind == "abs_terms":
            return s
        if kind == "drop_last_k":
            opa = a.T if ta else a
            opb = b.T if tb else b
            k = opa.shape[1]
            last = pam_ref.pam_mul_ref(opa[:, k - 1:k], opb[k - 1:k, :]).astype(np.float64)
            return c - last
        return c
    return gemm


@pytest.mark.parametrize("kind", ["square_b_read_untransposed", "swap_trans", "abs_terms", "drop_last_k"])
def test_gemm_mutant_is_caught(kind):
    assert caught(pins.GEMM_CHECKS, gemm_mutant(kind)) is not None, f"gemm mutant {kind} passed every pin"
