"""Seeded randomized parity sweep of the PAM matrix product against the C
oracle: random sizes (ragged in every dimension), transposes, batch counts,
padded leading dimensions and batch strides, every tile shape, random split
counts and whole-tile counts (hybrid plans), plus the library's own plan;
large outputs whose whole-K tiles span several rounds of resident
workgroups; then the same with narrow-mantissa and bfloat16 operands.  Each case is
compared element by element within the GEMM tolerance.  The environment
variable PAM_FUZZ_CASES sets the number of cases of the first sweep."""
import os

import numpy as np
import pytest

import paper_2305_17190_amd as pam
from gpu_util import check_gemm, device, note, oracle_gemm, to_dev
from oracle import pam_ref

pytestmark = pytest.mark.gpu

TILES = [(128, 128, 1), (128, 64, 1), (128, 64, 2), (64, 64, 1), (64, 64, 4)]
# PAM_FUZZ_CASES widens the sweep (same seeds first, then new ones).
CASES = int(os.environ.get("PAM_FUZZ_CASES", "1000"))


def draw(rng):
    m = int(rng.integers(1, 300))
    n = int(rng.integers(1, 300))
    k = int(rng.integers(1, 700))
    batch = int(rng.integers(1, 4))
    while m * n * k * batch > 6_000_000:
        k = max(1, k // 2)
    ta, tb = bool(rng.integers(0, 2)), bool(rng.integers(0, 2))
    pad = tuple(int(x) for x in rng.integers(0, 6, size=3))
    choice = int(rng.integers(0, 6))
    if choice == 0:
        plan = None                                        # the library's plan
    else:
        tm, tn, kg = TILES[int(rng.integers(0, len(TILES)))]
        splits = int(rng.integers(1, 9))
        tiles = -(-m // tm) * -(-n // tn) * batch
        whole = int(rng.integers(0, tiles + 1)) if choice >= 4 else 0
        plan = (tm, tn, splits, kg, whole)
    return m, n, k, batch, ta, tb, pad, plan


@pytest.mark.parametrize("case", range(CASES))
def test_random_products(case):
    import torch
    rng = np.random.default_rng(1000 + case)
    m, n, k, batch, ta, tb, pad, plan = draw(rng)
    a_rows, a_cols = (k, m) if ta else (m, k)
    b_rows, b_cols = (n, k) if tb else (k, n)
    lda, ldb, ldc = a_cols + pad[0], b_cols + pad[1], n + pad[2]
    # batch strides: whole padded matrices, plus a few spare rows
    sa, sb = (a_rows + 1) * lda, (b_rows + 2) * ldb
    a_buf = rng.standard_normal(batch * sa).astype(np.float32)
    b_buf = rng.standard_normal(batch * sb).astype(np.float32)
    if case % 3 == 0:                                      # zeros, denormals and tiny values
        for buf in (a_buf, b_buf):
            idx = rng.choice(buf.size, size=max(1, buf.size // 50), replace=False)
            buf[idx[0::3]] = 0.0
            buf[idx[1::3]] = np.float32(3e-41)
            buf[idx[2::3]] = np.float32(1.5e-38)
    note(f"fuzz {case}: m={m} n={n} k={k} batch={batch} ta={ta} tb={tb} pad={pad} plan={plan}")
    da = torch.as_strided(to_dev(a_buf), (batch, a_rows, a_cols), (sa, lda, 1))
    db = torch.as_strided(to_dev(b_buf), (batch, b_rows, b_cols), (sb, ldb, 1))
    c_full = torch.full((batch, m, ldc), float("nan"), device=device())
    c = c_full[:, :, :n]
    pam.bmm(da, db, trans_a=ta, trans_b=tb, out=c, plan=plan)
    got = c_full.cpu().numpy()
    assert np.all(np.isnan(got[:, :, n:])), "wrote outside the output's columns"
    c_ref, s_ref = oracle_gemm(a_buf, b_buf, ta, tb, m, n, k, lda, ldb, sa, sb, batches=list(range(batch)))
    check_gemm(got[:, :, :n], c_ref, s_ref, k, f"fuzz {case}")


# Resident workgroups of each tile shape on the 256 compute units.
SLOTS = {(128, 128, 1): 768, (128, 64, 1): 1024, (128, 64, 2): 512, (64, 64, 1): 2048, (64, 64, 4): 512}
LARGE_CASES = 30


@pytest.mark.parametrize("case", range(LARGE_CASES))
def test_random_large_products(case):
    # Outputs of 1000-4200 square, more tiles than resident workgroups, so
    # whole-K tiles span several rounds before the split ones (hybrid plans
    # whose whole-tile count is a multiple of the resident slots, as the
    # library plans them, or any count).  Compared in full with the C oracle.
    rng = np.random.default_rng(9000 + case)
    m, n = (int(x) for x in rng.integers(1000, 4200, size=2))
    k = int(rng.integers(16, 520))
    ta, tb = bool(rng.integers(0, 2)), bool(rng.integers(0, 2))
    tm, tn, kg = TILES[case % len(TILES)]
    tiles = -(-m // tm) * -(-n // tn)
    splits = int(rng.integers(1, 9))
    slots = SLOTS[(tm, tn, kg)]
    if case % 2 == 0 and tiles > slots:
        whole = slots * int(rng.integers(1, tiles // slots + 1))
        whole = min(whole, tiles - 1)
    else:
        whole = int(rng.integers(0, tiles + 1))
    plan = (tm, tn, splits, kg, whole)
    a_rows, a_cols = (k, m) if ta else (m, k)
    b_rows, b_cols = (n, k) if tb else (k, n)
    a_buf = rng.standard_normal(a_rows * a_cols).astype(np.float32)
    b_buf = rng.standard_normal(b_rows * b_cols).astype(np.float32)
    if case % 3 == 0:                                      # zeros, denormals and tiny values
        for buf in (a_buf, b_buf):
            idx = rng.choice(buf.size, size=max(1, buf.size // 500), replace=False)
            buf[idx[0::3]] = 0.0
            buf[idx[1::3]] = np.float32(3e-41)
            buf[idx[2::3]] = np.float32(1.5e-38)
    note(f"fuzz large {case}: m={m} n={n} k={k} ta={ta} tb={tb} plan={plan} tiles={tiles}")
    da = to_dev(a_buf).view(1, a_rows, a_cols)
    db = to_dev(b_buf).view(1, b_rows, b_cols)
    got = pam.bmm(da, db, trans_a=ta, trans_b=tb, plan=plan).cpu().numpy()
    c_ref, s_ref = oracle_gemm(a_buf, b_buf, ta, tb, m, n, k, a_cols, b_cols, batches=[0])
    check_gemm(got, c_ref, s_ref, k, f"fuzz large {case}")


NARROW_CASES = 200


@pytest.mark.parametrize("case", range(NARROW_CASES))
def test_random_narrow_and_bfloat16_products(case):
    # The same random sizes, transposes and padded layouts with operands of
    # fewer mantissa bits: float32 elements rounded to 0-10 mantissa bits by
    # the kernels, or bfloat16 elements widened exactly as they are loaded.
    # The oracle takes the rounded (resp. widened) float32 values.
    import torch
    rng = np.random.default_rng(5000 + case)
    m, n, k, batch, ta, tb, pad, _ = draw(rng)
    bf16 = case % 2 == 1
    bits = 7 if bf16 else int(rng.choice([0, 3, 4, 7, 10]))
    a_rows, a_cols = (k, m) if ta else (m, k)
    b_rows, b_cols = (n, k) if tb else (k, n)
    lda, ldb = a_cols + pad[0], b_cols + pad[1]
    sa, sb = (a_rows + 1) * lda, (b_rows + 2) * ldb
    a_buf = rng.standard_normal(batch * sa).astype(np.float32)
    b_buf = (rng.standard_normal(batch * sb) * 0.1).astype(np.float32)
    if case % 4 < 2:                                       # zeros, denormals and tiny values
        for buf in (a_buf, b_buf):
            idx = rng.choice(buf.size, size=max(1, buf.size // 50), replace=False)
            buf[idx[0::3]] = 0.0
            buf[idx[1::3]] = np.float32(3e-39)
            buf[idx[2::3]] = np.float32(1.5e-38)
    note(f"fuzz narrow {case}: m={m} n={n} k={k} batch={batch} ta={ta} tb={tb} pad={pad} "
         f"{'bfloat16' if bf16 else f'bits={bits}'}")
    if bf16:
        a16 = torch.from_numpy(a_buf).to(torch.bfloat16)
        b16 = torch.from_numpy(b_buf).to(torch.bfloat16)
        a_ref = (a16.view(torch.int16).numpy().view(np.uint16).astype(np.uint32) << 16).view(np.float32)
        b_ref = (b16.view(torch.int16).numpy().view(np.uint16).astype(np.uint32) << 16).view(np.float32)
        da, db = a16.to(device()), b16.to(device())
    else:
        a_ref, b_ref = pam_ref.round_mantissa_ref(a_buf, bits), pam_ref.round_mantissa_ref(b_buf, bits)
        da, db = to_dev(a_buf), to_dev(b_buf)
    da = torch.as_strided(da, (batch, a_rows, a_cols), (sa, lda, 1))
    db = torch.as_strided(db, (batch, b_rows, b_cols), (sb, ldb, 1))
    c = pam.bmm(da, db, trans_a=ta, trans_b=tb, mantissa_bits=bits).cpu().numpy()
    c_ref, s_ref = oracle_gemm(a_ref, b_ref, ta, tb, m, n, k, lda, ldb, sa, sb, batches=list(range(batch)))
    check_gemm(c, c_ref, s_ref, k, f"fuzz narrow {case}")
