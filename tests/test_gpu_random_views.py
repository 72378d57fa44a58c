"""Seeded random operand views of the batched product against the oracle.

Beside the randomized sweep of sizes and plans, each case here places its
operands at a storage offset (often not 16-byte aligned, so the kernels load
those operands element by element), leaves gaps between the matrices of a
batch, pads leading dimensions and the output's rows, and mixes float32 and
bfloat16 elements, normal values and planted zeros, denormals and tiny
normals, the library's plan and forced plans (tile shape, split count,
whole-K tile count).  The product must agree with the oracle within the GEMM
tolerance and leave the output's padding untouched; bfloat16 products must
equal the float32 product of the widened operands bit for bit.
"""
import numpy as np
import pytest

import paper_2305_17190_amd as pam
from gpu_util import check_gemm, device, note, oracle_gemm

pytestmark = pytest.mark.gpu

TILES = [(128, 128, 1), (128, 64, 1), (128, 64, 2), (64, 64, 1), (64, 64, 4)]


def draw(seed):
    g = np.random.default_rng(9100 + seed)
    dim = lambda: int(g.integers(1, 48)) if g.random() < 0.3 else int(g.integers(48, 330))
    m, n, k = dim(), dim(), int(g.integers(1, 40)) if g.random() < 0.2 else int(g.integers(40, 700))
    batch = int(g.integers(1, 4))
    while m * n * k * batch > 60_000_000:
        k = max(1, k // 2)
    c = dict(m=m, n=n, k=k, batch=batch, ta=bool(g.random() < 0.5), tb=bool(g.random() < 0.5),
             pad_a=int(g.integers(0, 10)) if g.random() < 0.5 else 0,
             pad_b=int(g.integers(0, 10)) if g.random() < 0.5 else 0,
             pad_c=int(g.integers(0, 6)) if g.random() < 0.3 else 0,
             gap=int(g.integers(1, 40)) if g.random() < 0.3 else 0,           # extra elements between matrices
             off_a=int(g.integers(0, 9)) if g.random() < 0.3 else 0,          # storage offset in elements
             off_b=int(g.integers(0, 9)) if g.random() < 0.3 else 0,
             bf16=bool(g.random() < 0.3), low=bool(g.random() < 0.4), plan=None)
    if not c["bf16"] and g.random() < 0.5:
        tm, tn, kg = TILES[int(g.integers(0, len(TILES)))]
        splits = int(g.choice([1, 2, 3, 5, 8]))
        tiles = -(-m // tm) * -(-n // tn) * batch
        whole = int(g.integers(0, tiles)) if splits > 1 and g.random() < 0.5 else 0
        c["plan"] = (tm, tn, splits, kg, whole)
    return c


def values(g, size, low):
    x = g.standard_normal(size).astype(np.float32)
    if low:
        r = g.random(size)
        x[r < 0.02] = 0.0
        x[(r >= 0.02) & (r < 0.03)] = np.float32(-3e-40)                   # denormal
        x[(r >= 0.03) & (r < 0.05)] = (g.uniform(1.0, 3.0, int(((r >= 0.03) & (r < 0.05)).sum())) *
                                       2.0 ** -120).astype(np.float32)      # tiny normals
    return x


def operand(g, batch, rows, cols, pad, gap, off, low, bf16):
    """A (batch, rows, cols) view with row stride cols + pad and matrix stride
    rows * (cols + pad) + gap, `off` elements into its storage; returns the
    device view and the float32 values of its storage from the view's first
    element (bfloat16 storage widened exactly)."""
    import torch
    ld = cols + pad
    stride = rows * ld + gap
    size = off + (batch - 1) * stride + rows * ld
    host = values(g, size, low)
    if bf16:
        t = torch.from_numpy(host).to(torch.bfloat16)
        flat = (t.view(torch.int16).numpy().view(np.uint16).astype(np.uint32) << 16).view(np.float32)
    else:
        t = torch.from_numpy(host)
        flat = host
    dev = t.to(device())
    view = dev[off:].as_strided((batch, rows, cols), (stride, ld, 1))
    return view, flat[off:], ld, stride


@pytest.mark.parametrize("seed", range(200))
def test_random_view(seed):
    import torch
    c = draw(seed)
    note(f"random view {seed}: {c}")
    g = np.random.default_rng(9500 + seed)
    m, n, k, batch, ta, tb = c["m"], c["n"], c["k"], c["batch"], c["ta"], c["tb"]
    a_rows, a_cols = (k, m) if ta else (m, k)
    b_rows, b_cols = (n, k) if tb else (k, n)
    A, a_flat, lda, sa = operand(g, batch, a_rows, a_cols, c["pad_a"], c["gap"], c["off_a"], c["low"], c["bf16"])
    B, b_flat, ldb, sb = operand(g, batch, b_rows, b_cols, c["pad_b"], c["gap"], c["off_b"], c["low"], c["bf16"])
    ldc = n + c["pad_c"]
    c_full = torch.full((batch, m, ldc), float("nan"), device=device())
    out = c_full[:, :, :n]
    pam.bmm(A, B, trans_a=ta, trans_b=tb, out=out, plan=c["plan"])
    got = c_full.cpu().numpy()
    if c["pad_c"]:
        assert np.all(np.isnan(got[:, :, n:])), "wrote outside the output's columns"
    c_ref, s_ref = oracle_gemm(a_flat, b_flat, ta, tb, m, n, k, lda, ldb, sa, sb, batches=list(range(batch)))
    check_gemm(got[:, :, :n], c_ref, s_ref, k, f"random view {seed}")
    if c["bf16"]:
        wide = pam.bmm(A.float(), B.float(), trans_a=ta, trans_b=tb)
        assert torch.equal(out.contiguous().view(torch.int32), wide.view(torch.int32)), \
            "bfloat16 product differs from the float32 product of the widened operands"
