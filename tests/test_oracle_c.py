"""The plain C oracle against the pins and against the Python oracle (CPU only)."""
import numpy as np
import pytest

import pam_workloads as wl
import pins
from oracle import pam_c, pam_ref


@pytest.fixture(scope="module", autouse=True)
def built():
    pam_c.build()
    pam_c.load()


def c_mul(a, b):
    a, b = np.broadcast_arrays(np.asarray(a, dtype=np.float32), np.asarray(b, dtype=np.float32))
    return pam_c.pam_mul(a.copy(), b.copy()).reshape(a.shape)


def c_gemm(a, b, ta, tb):
    opa_shape = a.shape[::-1] if ta else a.shape
    opb_shape = b.shape[::-1] if tb else b.shape
    m, k = opa_shape
    n = opb_shape[1]
    c, _ = pam_c.pam_gemm(a, b, ta, tb, m, n, k, a.shape[1], b.shape[1])
    return c[0]


@pytest.mark.parametrize("check", pins.SCALAR_CHECKS, ids=lambda c: c.__name__)
def test_c_scalar_pins(check):
    check(c_mul)


@pytest.mark.parametrize("check", pins.GEMM_CHECKS, ids=lambda c: c.__name__)
def test_c_gemm_pins(check):
    check(c_gemm)


def test_c_matches_python_elementwise():
    sp = wl.special_bit_patterns()
    a, b = np.meshgrid(sp, sp, indexing="ij")
    assert np.array_equal(c_mul(a, b).view(np.uint32), pam_ref.pam_mul_ref(a, b).view(np.uint32))
    r = wl.random_bit_patterns(1 << 18, 21)
    x, y = r[: 1 << 17], r[1 << 17:]
    assert np.array_equal(c_mul(x, y).view(np.uint32), pam_ref.pam_mul_ref(x, y).view(np.uint32))
    a1, b1 = wl.pam_mul_inputs(100003, 22)
    assert np.array_equal(c_mul(a1, b1).view(np.uint32), pam_ref.pam_mul_ref(a1, b1).view(np.uint32))


@pytest.mark.parametrize("ta,tb", [(False, False), (False, True), (True, False), (True, True)])
def test_c_matches_python_gemm(ta, tb):
    g = np.random.default_rng(int(ta) * 2 + int(tb))
    m, n, k = 37, 29, 53
    a_op = g.standard_normal((m, k)).astype(np.float32)
    b_op = g.standard_normal((k, n)).astype(np.float32)
    a_op[3, :] = 0.0
    b_op[:, 5] = np.float32(1e-39)
    a = np.ascontiguousarray(a_op.T) if ta else a_op
    b = np.ascontiguousarray(b_op.T) if tb else b_op
    c_py, s_py = pam_ref.pam_gemm_ref(a, b, ta, tb)
    c_c, s_c = pam_c.pam_gemm(a, b, ta, tb, m, n, k, a.shape[1], b.shape[1])
    assert np.array_equal(c_c[0], c_py)
    assert np.array_equal(s_c[0], s_py)


def test_c_batched_strided_subgrid():
    g = np.random.default_rng(9)
    batch, m, n, k = 4, 12, 10, 15
    a = g.standard_normal((batch, m, k)).astype(np.float32)
    b = g.standard_normal((batch, n, k)).astype(np.float32)           # trans_b layout
    rows, cols, bats = [0, 11, 5], [9, 0], [3, 1]
    c, s = pam_c.pam_gemm(a, b, False, True, m, n, k, k, k, m * k, n * k, batches=bats, rows=rows, cols=cols)
    for zi, z in enumerate(bats):
        cz, sz = pam_ref.pam_gemm_ref(a[z], b[z], False, True, rows=rows, cols=cols)
        assert np.array_equal(c[zi], cz)
        assert np.array_equal(s[zi], sz)


def test_c_uses_threads():
    assert pam_c.num_threads() >= 1
