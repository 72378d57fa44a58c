"""Elementwise pam_mul on the GPU: bit-exact against the CPU oracle."""
import numpy as np
import pytest

import pam_workloads as wl
import paper_2305_17190_amd as pam
from gpu_util import device, note, to_dev
from oracle import pam_c, pam_ref

pytestmark = pytest.mark.gpu


def run(a, b):
    out = pam.mul(to_dev(a), to_dev(b))
    return out.cpu().numpy()


def assert_bits_equal(got, want, what):
    g = got.view(np.uint32)
    w = want.view(np.uint32)
    bad = np.nonzero(g != w)[0]
    assert bad.size == 0, (f"{what}: {bad.size} mismatches, first at {bad[0]}: "
                           f"got {g[bad[0]]:#010x} want {w[bad[0]]:#010x}")


def test_workload1_elementwise_million():
    note("pam_mul 2^20 elements, workload 1 inputs")
    a, b = wl.pam_mul_inputs(1 << 20, 1000 + 3)
    assert_bits_equal(run(a, b), pam_c.pam_mul(a, b), "2^20")


def test_special_pattern_cross_product():
    note("pam_mul special patterns cross product")
    sp = wl.special_bit_patterns()
    a, b = np.meshgrid(sp, sp, indexing="ij")
    a = a.reshape(-1).copy()
    b = b.reshape(-1).copy()
    assert_bits_equal(run(a, b), pam_ref.pam_mul_ref(a, b), "special cross product")


def test_random_bit_patterns_16m():
    note("pam_mul 2^24 random bit-pattern pairs")
    r = wl.random_bit_patterns(1 << 25, 4242)
    a, b = r[: 1 << 24].copy(), r[1 << 24:].copy()
    assert_bits_equal(run(a, b), pam_c.pam_mul(a, b), "random bits")


@pytest.mark.parametrize("n", [1, 3, 4, 5, 255, 1023, (1 << 20) + 3])
def test_tail_sizes(n):
    note(f"pam_mul n={n}")
    a, b = wl.pam_mul_inputs(n, 77 + n)
    assert_bits_equal(run(a, b), pam_ref.pam_mul_ref(a, b), f"n={n}")


def test_unaligned_views_use_scalar_path():
    note("pam_mul unaligned views")
    a, b = wl.pam_mul_inputs(10001, 5)
    da, db = to_dev(a), to_dev(b)
    out = pam.mul(da[1:], db[1:])
    assert_bits_equal(out.cpu().numpy(), pam_ref.pam_mul_ref(a[1:], b[1:]), "offset 1")


def test_in_place():
    note("pam_mul in place")
    a, b = wl.pam_mul_inputs(4097, 6)
    da, db = to_dev(a), to_dev(b)
    pam.mul(da, db, out=da)
    assert_bits_equal(da.cpu().numpy(), pam_ref.pam_mul_ref(a, b), "in place")


def test_empty():
    import torch
    e = torch.empty(0, device=device())
    assert pam.mul(e, e).numel() == 0


def test_repeatable_and_stream_ordered():
    import torch
    note("pam_mul on a side stream")
    a, b = wl.pam_mul_inputs(1 << 16, 8)
    da, db = to_dev(a), to_dev(b)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        o1 = pam.mul(da, db)
        o2 = pam.mul(da, db)
    s.synchronize()
    assert torch.equal(o1.view(torch.int32), o2.view(torch.int32))
    assert_bits_equal(o1.cpu().numpy(), pam_ref.pam_mul_ref(a, b), "side stream")
