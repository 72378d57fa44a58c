"""Checks that pin an implementation of R11's rounding to m mantissa bits
(App. "PAM with Narrower Mantissas") to library conversions, exact rationals
and invariants.  Each check takes ``rnd(x, bits)`` (float32 array in, float32
array out), so the same checks run on the oracle, on planted mistakes and on
the HIP kernel."""
from fractions import Fraction

import numpy as np
import pytest

SIGN, INF = 0x80000000, 0x7F800000


def bits(x):
    return np.asarray(x, np.float32).view(np.uint32)


def sample(n, seed):
    g = np.random.default_rng(seed)
    u = g.integers(0, 1 << 32, size=n, dtype=np.uint64).astype(np.uint32)
    near = np.array([0x3F7FFFFF, 0x3FFFFFFF, 0x7F7FFFFF, 0xFF7FFFFF, 0x007FFFFF, 0x00000001, 0x3F808000,
                     0x3F818000, 0x3F80C000, 0x7F800000, 0xFF800000, 0x00800000], dtype=np.uint32)
    return np.concatenate([near, u]).view(np.float32)


def value(u):
    s, ex, fr = u >> 31, (u >> 23) & 0xFF, u & 0x7FFFFF
    v = Fraction(fr, 1 << 23) * Fraction(2) ** -126 if ex == 0 else (1 + Fraction(fr, 1 << 23)) * Fraction(2) ** (ex - 127)
    return -v if s else v


def check_bf16(rnd):
    """bits = 7 is bfloat16: torch's float32 -> bfloat16 conversion (nearest even)."""
    torch = pytest.importorskip("torch")
    x = sample(50000, 1)
    x = x[~np.isnan(x)]
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(bits(rnd(x, 7)), bits(want))


def check_fp16_range(rnd):
    """bits = 10 is float16's mantissa: numpy's float32 -> float16 conversion on
    float16's normal range."""
    g = np.random.default_rng(2)
    x = (g.uniform(-1, 1, size=50000) * np.exp2(g.integers(-14, 15, size=50000))).astype(np.float32)
    x = x[(np.abs(x) >= 2.0 ** -14) & (np.abs(x) <= 65504)]
    assert np.array_equal(bits(rnd(x, 10)), bits(x.astype(np.float16).astype(np.float32)))


def check_nearest_on_the_grid(rnd):
    """The result has at most `bits` mantissa bits and is the nearest such value
    (ties to even), checked against its two grid neighbours in exact rationals."""
    x = sample(3000, 3)
    for b in (0, 1, 3, 4, 7, 15):
        y = bits(rnd(x, b))
        drop = 23 - b
        for xu, yu in zip(bits(x), y):
            xu, yu = int(xu), int(yu)
            if (xu & INF) == INF:
                assert yu == xu
                continue
            if (yu & INF) == INF:                      # rounded past FLT_MAX
                assert (xu & 0x7FFFFFFF) > 0x7F7FFFFF - (1 << (drop - 1)) if drop else False
                continue
            assert yu & ((1 << drop) - 1) == 0, (hex(xu), b, hex(yu))
            assert (yu >> 31) == (xu >> 31) or (yu & 0x7FFFFFFF) == 0
            q = abs(value(xu))
            v = abs(value(yu))
            step = 1 << drop
            for nb in ((yu & 0x7FFFFFFF) - step, (yu & 0x7FFFFFFF) + step):
                if nb < 0 or (nb & INF) == INF:
                    continue
                d, dn = abs(v - q), abs(value(nb) - q)
                assert d < dn or (d == dn and ((yu >> drop) & 1) == 0), (hex(xu), b, hex(yu))


def check_invariants(rnd):
    x = sample(20000, 4)
    fin = ~np.isnan(x)
    assert np.array_equal(bits(rnd(x, 23)), bits(x))
    for b in (0, 3, 7):
        y = rnd(x, b)
        assert np.array_equal(bits(rnd(y, b))[fin], bits(y)[fin])                # idempotent
        assert np.array_equal(bits(rnd(-x, b))[fin], bits(y)[fin] ^ SIGN)        # odd
        xs = np.sort(x[fin & np.isfinite(x)])
        ys = rnd(xs, b).astype(np.float64)
        assert np.all(ys[1:] >= ys[:-1])                                          # monotone
    assert np.all(np.isnan(rnd(np.float32([np.nan]), 3)))


CHECKS = [check_bf16, check_fp16_range, check_nearest_on_the_grid, check_invariants]


