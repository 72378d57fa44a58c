"""The CPU oracle against what the paper fixes (no GPU needed)."""
import numpy as np
import pytest

import pins
from oracle import pam_ref


def oracle_gemm(a, b, ta, tb):
    return pam_ref.pam_gemm_ref(a, b, ta, tb)[0]


def scalar_bits_vec(fn):
    """Lift a scalar bits -> bits function to float32 arrays."""
    def mul(a, b):
        a = np.asarray(a, dtype=np.float32)
        b = np.asarray(b, dtype=np.float32)
        a, b = np.broadcast_arrays(a, b)
        ua = a.view(np.uint32).reshape(-1)
        ub = b.view(np.uint32).reshape(-1)
        out = np.fromiter((fn(int(x), int(y)) for x, y in zip(ua, ub)), dtype=np.uint32, count=ua.size)
        return out.view(np.float32).reshape(a.shape)
    return mul


@pytest.mark.parametrize("check", pins.SCALAR_CHECKS, ids=lambda c: c.__name__)
def test_vectorised_bit_form(check):
    check(pam_ref.pam_mul_ref)


FAST_SCALAR = [pins.check_golden, pins.check_max_error_example, pins.check_range_readings,
               pins.check_symmetries, pins.check_error_bounds, pins.check_value_form]


@pytest.mark.parametrize("check", FAST_SCALAR, ids=lambda c: c.__name__)
def test_scalar_bit_form(check):
    check(scalar_bits_vec(pam_ref.pam_bits))


@pytest.mark.parametrize("check", FAST_SCALAR, ids=lambda c: c.__name__)
def test_scalar_field_form(check):
    check(scalar_bits_vec(pam_ref.pam_fields))


def test_three_forms_agree_on_random_and_special_patterns():
    """Bit form (int add), field form (Sec. 2.2 equations) and value form (Sec. 2.3)."""
    import pam_workloads as wl
    sp = wl.special_bit_patterns().view(np.uint32)
    rnd = wl.random_bit_patterns(20000, 7).view(np.uint32)
    pairs = [(int(x), int(y)) for x in sp for y in sp]
    pairs += list(zip(map(int, rnd[:10000]), map(int, rnd[10000:])))
    for ua, ub in pairs:
        rb = pam_ref.pam_bits(ua, ub)
        rf = pam_ref.pam_fields(ua, ub)
        assert rb == rf, (hex(ua), hex(ub), hex(rb), hex(rf))
        ea, eb = (ua >> 23) & 0xFF, (ub >> 23) & 0xFF
        if 0 < ea < 255 and 0 < eb < 255:
            a = float(np.uint32(ua).view(np.float32))
            b = float(np.uint32(ub).view(np.float32))
            v = np.float32(pam_ref.pam_value(a, b)).view(np.uint32)
            assert int(v) == rb, (hex(ua), hex(ub), hex(rb), hex(int(v)))


def test_vectorised_matches_scalar_on_all_special_pairs():
    import pam_workloads as wl
    sp = wl.special_bit_patterns()
    a, b = np.meshgrid(sp, sp, indexing="ij")
    got = pam_ref.pam_mul_ref(a, b).view(np.uint32)
    for i in range(a.shape[0]):
        for j in range(a.shape[1]):
            want = pam_ref.pam_bits(int(a[i, j].view(np.uint32)), int(b[i, j].view(np.uint32)))
            assert int(got[i, j]) == want


@pytest.mark.parametrize("check", pins.GEMM_CHECKS, ids=lambda c: c.__name__)
def test_gemm_oracle(check):
    check(oracle_gemm)


def test_gemm_outer_product():
    pins.check_gemm_outer(oracle_gemm, pam_ref.pam_mul_ref)


def test_gemm_sum_of_abs_and_tolerance():
    g = np.random.default_rng(3)
    a = g.standard_normal((6, 9)).astype(np.float32)
    b = g.standard_normal((9, 4)).astype(np.float32)
    c, s = pam_ref.pam_gemm_ref(a, b)
    terms = pam_ref.pam_mul_ref(a[:, :, None], b[None, :, :]).astype(np.float64)
    assert np.allclose(s, np.abs(terms).sum(axis=1), rtol=1e-15, atol=0)
    assert np.all(np.abs(c) <= s)
    tol = pam_ref.gemm_tolerance(s, 9)
    assert np.all(tol > 0)


def test_gemm_batched_powers_of_two():
    g = np.random.default_rng(5)
    a = g.standard_normal((3, 5, 7)).astype(np.float32)
    e = g.integers(-4, 5, size=(3, 7, 6))
    b = np.ldexp(1.0, e).astype(np.float32)
    c, _ = pam_ref.pam_gemm_batched_ref(a, b)
    assert np.allclose(c, a.astype(np.float64) @ b.astype(np.float64), rtol=1e-12, atol=1e-12)
    c_t, _ = pam_ref.pam_gemm_batched_ref(np.ascontiguousarray(a.transpose(0, 2, 1)), b, trans_a=True)
    assert np.array_equal(c, c_t)


def test_gemm_subgrid_matches_full():
    g = np.random.default_rng(6)
    a = g.standard_normal((10, 8)).astype(np.float32)
    b = g.standard_normal((8, 9)).astype(np.float32)
    c, s = pam_ref.pam_gemm_ref(a, b)
    rows, cols = [7, 2, 9], [0, 8, 3, 3]
    c2, s2 = pam_ref.pam_gemm_ref(a, b, rows=rows, cols=cols)
    assert np.array_equal(c2, c[np.ix_(rows, cols)])
    assert np.array_equal(s2, s[np.ix_(rows, cols)])
