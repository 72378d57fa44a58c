"""The PAD / palog2 / paexp2 oracle against the paper's facts (tests/pa_pins.py),
and its bit / field / exact-rational renderings against each other."""
import numpy as np
import pytest

import pa_pins
from oracle import pa_ref, pam_ref


@pytest.mark.parametrize("check", pa_pins.PAD_CHECKS, ids=lambda c: c.__name__)
def test_pad_pins(check):
    check(pa_ref.pad_ref)


def test_pad_inverts_pam():
    pa_pins.check_pad_inverts_pam(pa_ref.pad_ref, pam_ref.pam_mul_ref)


@pytest.mark.parametrize("check", pa_pins.PALOG2_CHECKS, ids=lambda c: c.__name__)
def test_palog2_pins(check):
    check(pa_ref.palog2_ref)


@pytest.mark.parametrize("check", pa_pins.PAEXP2_CHECKS, ids=lambda c: c.__name__)
def test_paexp2_pins(check):
    check(pa_ref.paexp2_ref)


def specials():
    vals = [0x00000000, 0x80000000, 0x00000001, 0x807FFFFF, 0x00800000, 0x80800000, 0x3F800000, 0xBF800000,
            0x3FC00000, 0xC0400000, 0x7F7FFFFF, 0xFF7FFFFF, 0x7F800000, 0xFF800000, 0x7FC00000, 0xFFC00000,
            0x7F800001, 0x1F800000, 0x5F800000, 0x20000000, 0x5F000000, 0x42FE0000, 0xC2FC0000, 0x43000000,
            0xC3000000, 0x33800000, 0xB3800000, 0x34400000]
    return np.array(vals, dtype=np.uint32)


def random_bits(n, seed):
    return np.random.default_rng(seed).integers(0, 1 << 32, size=n, dtype=np.uint64).astype(np.uint32)


def test_pad_bit_form_equals_field_form():
    s = specials()
    ua, ub = np.meshgrid(s, s, indexing="ij")
    ua = np.concatenate([ua.reshape(-1), random_bits(20000, 41)])
    ub = np.concatenate([ub.reshape(-1), random_bits(20000, 42)])
    vec = pa_pins.bits(pa_ref.pad_ref(pa_pins.f32(ua), pa_pins.f32(ub)))
    for x, y, v in zip(ua, ub, vec):
        assert pa_ref.pad_bits(int(x), int(y)) == int(v) == pa_ref.pad_fields(int(x), int(y)), (hex(x), hex(y))


def test_palog2_vector_equals_exact_rational():
    u = np.concatenate([specials(), random_bits(20000, 43)])
    vec = pa_pins.bits(pa_ref.palog2_ref(pa_pins.f32(u)))
    for x, v in zip(u, vec):
        assert pa_ref.palog2_exact(int(x)) == int(v), hex(x)


def test_paexp2_vector_equals_exact_rational():
    g = np.random.default_rng(44)
    near = (g.uniform(-140, 140, size=20000)).astype(np.float32).view(np.uint32)
    small = ((g.integers(0, 2, size=5000) << 31) | (g.integers(60, 127, size=5000) << 23)
             | g.integers(0, 1 << 23, size=5000)).astype(np.uint32)
    u = np.concatenate([specials(), random_bits(5000, 45), near, small])
    vec = pa_pins.bits(pa_ref.paexp2_ref(pa_pins.f32(u)))
    for x, v in zip(u, vec):
        assert pa_ref.paexp2_exact(int(x)) == int(v), hex(x)
