"""Elementwise PAD, palog2 and paexp2 on the GPU: bit-exact against the CPU
oracle, and held to the same pins as the oracle (tests/pa_pins.py)."""
import numpy as np
import pytest

import pa_pins
import pam_workloads as wl
import paper_2305_17190_amd as pam
from gpu_util import device, note, to_dev
from oracle import pa_ref, pam_ref

pytestmark = pytest.mark.gpu


def gpu_pad(a, b):
    a, b = np.broadcast_arrays(np.asarray(a, np.float32), np.asarray(b, np.float32))
    shape = a.shape
    return pam.pad(to_dev(a.reshape(-1)), to_dev(b.reshape(-1))).cpu().numpy().reshape(shape)


def gpu_palog2(a):
    a = np.asarray(a, np.float32)
    return pam.palog2(to_dev(a.reshape(-1))).cpu().numpy().reshape(a.shape)


def gpu_paexp2(a):
    a = np.asarray(a, np.float32)
    return pam.paexp2(to_dev(a.reshape(-1))).cpu().numpy().reshape(a.shape)


def gpu_mul(a, b):
    a, b = np.broadcast_arrays(np.asarray(a, np.float32), np.asarray(b, np.float32))
    return pam.mul(to_dev(a.reshape(-1)), to_dev(b.reshape(-1))).cpu().numpy().reshape(a.shape)


def assert_bits_equal(got, want, what):
    g = np.asarray(got, np.float32).view(np.uint32).reshape(-1)
    w = np.asarray(want, np.float32).view(np.uint32).reshape(-1)
    bad = np.nonzero(g != w)[0]
    assert bad.size == 0, (f"{what}: {bad.size} mismatches, first at {bad[0]}: "
                           f"got {g[bad[0]]:#010x} want {w[bad[0]]:#010x}")


@pytest.mark.parametrize("check", pa_pins.PAD_CHECKS, ids=lambda c: c.__name__)
def test_pad_pins_on_gpu(check):
    note(f"pad pin {check.__name__}")
    check(gpu_pad)


def test_pad_inverts_pam_on_gpu():
    note("pad inverts pam (both on the GPU)")
    pa_pins.check_pad_inverts_pam(gpu_pad, gpu_mul)


@pytest.mark.parametrize("check", pa_pins.PALOG2_CHECKS, ids=lambda c: c.__name__)
def test_palog2_pins_on_gpu(check):
    note(f"palog2 pin {check.__name__}")
    check(gpu_palog2)


@pytest.mark.parametrize("check", pa_pins.PAEXP2_CHECKS, ids=lambda c: c.__name__)
def test_paexp2_pins_on_gpu(check):
    note(f"paexp2 pin {check.__name__}")
    check(gpu_paexp2)


def test_pad_special_cross_product():
    note("pad special patterns cross product")
    sp = wl.special_bit_patterns()
    a, b = np.meshgrid(sp, sp, indexing="ij")
    a, b = a.reshape(-1).copy(), b.reshape(-1).copy()
    assert_bits_equal(gpu_pad(a, b), pa_ref.pad_ref(a, b), "special cross product")


def test_pad_random_bits_and_normal_inputs():
    note("pad 2^22 random bit-pattern pairs and 2^20 N(0,1) pairs")
    r = wl.random_bit_patterns(1 << 23, 5151)
    a, b = r[: 1 << 22].copy(), r[1 << 22:].copy()
    assert_bits_equal(gpu_pad(a, b), pa_ref.pad_ref(a, b), "random bits")
    a, b = wl.pam_mul_inputs(1 << 20, 5152)
    assert_bits_equal(gpu_pad(a, b), pa_ref.pad_ref(a, b), "N(0,1) with zeros and powers of two")


@pytest.mark.parametrize("fn,ref", [(gpu_palog2, pa_ref.palog2_ref), (gpu_paexp2, pa_ref.paexp2_ref)],
                         ids=["palog2", "paexp2"])
def test_unary_random_bits_and_specials(fn, ref):
    note(f"{fn.__name__} 2^22 random bit patterns and specials")
    x = np.concatenate([wl.special_bit_patterns(), wl.random_bit_patterns(1 << 22, 5253)])
    assert_bits_equal(fn(x), ref(x), "random bits")


def test_paexp2_softmax_shaped_arguments():
    note("paexp2 on 2^20 softmax-shaped arguments")
    x = wl.paexp2_arguments(1 << 20, 5354)
    assert_bits_equal(gpu_paexp2(x), pa_ref.paexp2_ref(x), "softmax-shaped")


def test_palog2_every_mantissa_of_three_octaves():
    note("palog2 on every mantissa of [2^-1, 2^2) and of [2^100, 2^101)")
    m = np.arange(1 << 23, dtype=np.uint32)
    for e in (126, 127, 128, 227):
        x = ((e << 23) | m).astype(np.uint32).view(np.float32)
        assert_bits_equal(gpu_palog2(x), pa_ref.palog2_ref(x), f"octave {e - 127}")


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 257, 4099])
def test_tail_sizes(n):
    note(f"pad / palog2 / paexp2 n={n}")
    a, b = wl.pam_mul_inputs(n, 90 + n)
    assert_bits_equal(gpu_pad(a, b), pa_ref.pad_ref(a, b), f"pad n={n}")
    assert_bits_equal(gpu_palog2(np.abs(a)), pa_ref.palog2_ref(np.abs(a)), f"palog2 n={n}")
    assert_bits_equal(gpu_paexp2(a * 10), pa_ref.paexp2_ref(a * 10), f"paexp2 n={n}")


def test_unaligned_views_and_in_place():
    note("pad / palog2 / paexp2 unaligned views and in place")
    a, b = wl.pam_mul_inputs(10001, 91)
    da, db = to_dev(a), to_dev(b)
    assert_bits_equal(pam.pad(da[1:], db[1:]).cpu().numpy(), pa_ref.pad_ref(a[1:], b[1:]), "pad offset 1")
    assert_bits_equal(pam.palog2(da[3:]).cpu().numpy(), pa_ref.palog2_ref(a[3:]), "palog2 offset 3")
    assert_bits_equal(pam.paexp2(da[2:]).cpu().numpy(), pa_ref.paexp2_ref(a[2:]), "paexp2 offset 2")
    pam.pad(da, db, out=da)
    assert_bits_equal(da.cpu().numpy(), pa_ref.pad_ref(a, b), "pad in place")
    pam.paexp2(db, out=db)
    assert_bits_equal(db.cpu().numpy(), pa_ref.paexp2_ref(b), "paexp2 in place")


def test_empty():
    import torch
    e = torch.empty(0, device=device())
    assert pam.pad(e, e).numel() == 0
    assert pam.palog2(e).numel() == 0
    assert pam.paexp2(e).numel() == 0


def test_pam_of_palog2_sum_matches_pam_for_unit_octave():
    """Sec. 2.3: for A, B in [1, 2), A .^ B = paexp2(palog2 A + palog2 B), and the
    palog2 values are exact there, so the GPU's three kernels must agree."""
    note("paexp2(palog2 a + palog2 b) == pam(a, b) on [1, 2)")
    g = np.random.default_rng(92)
    a = (0x3F800000 | g.integers(0, 1 << 23, size=1 << 16)).astype(np.uint32).view(np.float32)
    b = (0x3F800000 | g.integers(0, 1 << 23, size=1 << 16)).astype(np.uint32).view(np.float32)
    s = gpu_palog2(a) + gpu_palog2(b)     # exact: both in [0, 1) with 23 fraction bits
    assert_bits_equal(gpu_paexp2(s), pam_ref.pam_mul_ref(a, b), "composition")
