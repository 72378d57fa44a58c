"""Planted mistakes in copies of the PAD / palog2 / paexp2 oracle must be caught
by the pins of tests/pa_pins.py (each mutant by at least one pin).  Mutants
live here, on the CPU; the oracle itself is not modified."""
import numpy as np
import pytest

import pa_pins
from oracle import pa_ref, pam_ref

SIGN, MAG, BIAS = 0x80000000, 0x7FFFFFFF, 0x3F800000
MIN_NORMAL, FLT_MAX, INF, QNAN = 0x00800000, 0x7F7FFFFF, 0x7F800000, 0x7FC00000


def u64(x):
    return np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.int64)


def pad_variant(bias=BIAS, sign="xor", under="lt", over="flt_max", x_over_zero="inf", zero_over_zero="nan",
                swap=False, borrow="int"):
    def pad(a, b):
        a, b = np.broadcast_arrays(np.asarray(a, np.float32), np.asarray(b, np.float32))
        if swap:
            a, b = b, a
        ua, ub = u64(a), u64(b)
        s = ((ua ^ ub) if sign == "xor" else (ua | ub)) & SIGN
        ma, mb = ua & MAG, ub & MAG
        if borrow == "int":
            t = ma - mb + bias
        else:
            # field form with the printed conditions: E - 1{dM <= 0}, M + 1{dM <= 1}
            ea, eb = ma >> 23, mb >> 23
            fa, fb = ma & 0x7FFFFF, mb & 0x7FFFFF
            dm = fa - fb
            e = ea - eb + 127 - (dm <= 0)
            f = dm + (1 << 23) * (dm <= (1 << 23))
            t = (e << 23) + f
        small = (t < MIN_NORMAL) if under == "lt" else (t <= MIN_NORMAL)
        out = np.where(t > FLT_MAX, s | (FLT_MAX if over == "flt_max" else INF), s | (t & MAG))
        out = np.where(small, s, out)
        az, bz = ma < MIN_NORMAL, mb < MIN_NORMAL
        out = np.where(bz, s | INF if x_over_zero == "inf" else s, out)
        out = np.where(az, np.where(bz, QNAN if zero_over_zero == "nan" else s, s), out)
        out = np.where(mb == INF, s, out)
        out = np.where(ma == INF, np.where(mb == INF, QNAN, s | INF), out)
        out = np.where((ma > INF) | (mb > INF), QNAN, out)
        return out.astype(np.uint32).view(np.float32)
    return pad


PAD_MUTANTS = {
    "printed_borrow_conditions": pad_variant(borrow="printed"),
    "no_bias": pad_variant(bias=0),
    "bias_off_by_one_exponent": pad_variant(bias=126 << 23),
    "operands_swapped": pad_variant(swap=True),
    "sign_or": pad_variant(sign="or"),
    "underflow_off_by_one": pad_variant(under="le"),
    "overflow_to_inf": pad_variant(over="inf"),
    "x_over_zero_is_zero": pad_variant(x_over_zero="zero"),
    "zero_over_zero_is_zero": pad_variant(zero_over_zero="zero"),
}


def caught(checks, fn):
    for check in checks:
        try:
            check(fn)
        except AssertionError:
            return True
    return False


def test_oracle_passes_every_check():
    assert not caught(pa_pins.PAD_CHECKS, pa_ref.pad_ref)
    assert not caught(pa_pins.PALOG2_CHECKS, pa_ref.palog2_ref)
    assert not caught(pa_pins.PAEXP2_CHECKS, pa_ref.paexp2_ref)


@pytest.mark.parametrize("name", sorted(PAD_MUTANTS))
def test_pad_mutant_is_caught(name):
    fn = PAD_MUTANTS[name]
    checks = pa_pins.PAD_CHECKS + [lambda p: pa_pins.check_pad_inverts_pam(p, pam_ref.pam_mul_ref)]
    assert caught(checks, fn), f"no pin rejects PAD mutant {name}"


def palog2_variant(bias=BIAS, rounding="nearest", negative="nan", zero="-inf", mantissa=True):
    def palog2(a):
        a = np.asarray(a, np.float32)
        u = u64(a)
        mag = u & MAG
        num = (mag - bias) if mantissa else ((mag & 0x7F800000) - bias)
        v = num.astype(np.float64) / float(1 << 23)
        if rounding == "nearest":
            r = v.astype(np.float32)
        else:   # toward zero
            r = v.astype(np.float32)
            over = np.abs(r.astype(np.float64)) > np.abs(v)
            r = np.where(over, np.nextafter(r, np.float32(0)), r).astype(np.float32)
        out = r.view(np.uint32).astype(np.int64)
        zval = 0xFF800000 if zero == "-inf" else 0xC2FC0000
        out = np.where(mag < MIN_NORMAL, zval, out)
        if negative == "nan":
            out = np.where((u >= SIGN) & (mag >= MIN_NORMAL), QNAN, out)
        out = np.where(u == INF, INF, out)
        out = np.where(mag > INF, QNAN, out)
        return out.astype(np.uint32).view(np.float32)
    return palog2


PALOG2_MUTANTS = {
    "bias_off_by_one_exponent": palog2_variant(bias=126 << 23),
    "rounds_toward_zero": palog2_variant(rounding="zero"),
    "negative_uses_magnitude": palog2_variant(negative="abs"),
    "zero_gives_min_exponent": palog2_variant(zero="min"),
    "mantissa_dropped": palog2_variant(mantissa=False),
}


@pytest.mark.parametrize("name", sorted(PALOG2_MUTANTS))
def test_palog2_mutant_is_caught(name):
    assert caught(pa_pins.PALOG2_CHECKS, PALOG2_MUTANTS[name]), f"no pin rejects palog2 mutant {name}"


def paexp2_variant(bias=BIAS, rounding="even", floor="floor", over="inf", under="zero"):
    def paexp2(a):
        a = np.asarray(a, np.float32)
        u = u64(a)
        mag = u & MAG
        x = np.where(mag < MIN_NORMAL, 0.0, a.astype(np.float64))
        x = np.clip(np.nan_to_num(x, nan=0.0, posinf=256.0, neginf=-256.0), -256.0, 256.0)
        if floor == "trunc":
            # 2^trunc(A) (1 + A - trunc(A)): wrong for negative non-integers
            t = np.trunc(x)
            frac = x - t
            y = t * float(1 << 23) + frac * float(1 << 23)
            r = np.where(x < 0, np.rint(t * float(1 << 23) + np.abs(frac) * float(1 << 23)), np.rint(y))
        elif rounding == "even":
            r = np.rint(x * float(1 << 23))
        elif rounding == "half_up":
            r = np.floor(x * float(1 << 23) + 0.5)
        else:
            r = np.trunc(x * float(1 << 23))
        enc = r.astype(np.int64) + bias
        out = np.where(enc >= INF, INF if over == "inf" else FLT_MAX, enc)
        out = np.where(enc < MIN_NORMAL, 0 if under == "zero" else MIN_NORMAL, out)
        out = np.where(mag > INF, QNAN, out)
        return out.astype(np.uint32).view(np.float32)
    return paexp2


PAEXP2_MUTANTS = {
    "bias_off_by_one_exponent": paexp2_variant(bias=126 << 23),
    "ties_round_up": paexp2_variant(rounding="half_up"),
    "truncates_fraction": paexp2_variant(rounding="trunc"),
    "trunc_instead_of_floor": paexp2_variant(floor="trunc"),
    "overflow_to_flt_max": paexp2_variant(over="flt_max"),
    "underflow_to_min_normal": paexp2_variant(under="min"),
}


@pytest.mark.parametrize("name", sorted(PAEXP2_MUTANTS))
def test_paexp2_mutant_is_caught(name):
    assert caught(pa_pins.PAEXP2_CHECKS, PAEXP2_MUTANTS[name]), f"no pin rejects paexp2 mutant {name}"
