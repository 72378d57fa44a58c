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


EVERY_A_B = {
    "1.5": 0x3FC00000, "-1": 0xBF800000, "1.5*2^-63": 0x20400000, "FLT_MAX": 0x7F7FFFFF,
    "denormal": 0x00012345, "inf": 0x7F800000,
}


@pytest.mark.parametrize("name", list(EVERY_A_B))
def test_every_encoding_of_a(name):
    """All 2^32 float32 encodings of a against one fixed b (a carry-taking
    mantissa, a negative power of two, a value whose products cross both the
    underflow and the overflow boundary, the largest finite value, a
    denormal, inf), bit for bit against the C oracle, in chunks of 2^27,
    stopping at the first chunk that differs."""
    import torch
    ub = EVERY_A_B[name]
    note(f"pam_mul, every encoding of a, b = {name} ({ub:#010x})")
    chunk = 1 << 27
    bfull = np.full(chunk, ub, dtype=np.uint32).view(np.float32)
    bd = torch.full((chunk,), np.int32(np.uint32(ub).view(np.int32)), dtype=torch.int32,
                    device=device()).view(torch.float32)
    out = torch.empty(chunk, dtype=torch.float32, device=device())
    for c in range(1 << 5):
        a = np.arange(c * chunk, (c + 1) * chunk, dtype=np.uint64).astype(np.uint32).view(np.float32)
        pam.mul(to_dev(a), bd, out=out)
        got = out.cpu().numpy()
        want = pam_c.pam_mul(a, bfull)
        assert_bits_equal(got, want, f"b={name}, a encodings [{c * chunk:#x}, {(c + 1) * chunk:#x})")
