"""Helpers for the GPU parity tests: device transfer, HIP calls through the
C ABI binding, CPU-oracle references and the comparison rule."""
from __future__ import annotations

import sys
import warnings

import numpy as np
import pytest

from oracle import pam_c, pam_ref


def device():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        raise RuntimeError("GPU test run without a HIP device")
    return torch.device("cuda:0")


def note(msg: str) -> None:
    """Name the case on stdout before it touches the GPU."""
    sys.stdout.write(f"[case] {msg}\n")
    sys.stdout.flush()


def to_dev(x: np.ndarray):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to(device())


def oracle_gemm(a_buf, b_buf, ta, tb, m, n, k, lda, ldb, stride_a=0, stride_b=0, batches=None, rows=None,
                cols=None):
    """C and S from the C oracle over flat operand buffers (float64)."""
    return pam_c.pam_gemm(a_buf, b_buf, ta, tb, m, n, k, lda, ldb, stride_a, stride_b, batches, rows, cols)


def check_gemm(c_gpu: np.ndarray, c_ref: np.ndarray, s_ref: np.ndarray, k: int, what: str) -> None:
    """|C_gpu - C_ref| <= 1e-5 sqrt(K) S + K 2^-126, with NaN/inf positions equal.

    A float64 reference beyond the float32 range must come back as the same
    signed inf.
    """
    c = np.asarray(c_gpu, dtype=np.float64)
    assert c.shape == c_ref.shape, (what, c.shape, c_ref.shape)
    nan_r = np.isnan(c_ref)
    nan_g = np.isnan(c)
    assert np.array_equal(nan_r, nan_g), f"{what}: NaN positions differ ({nan_r.sum()} ref vs {nan_g.sum()} gpu)"
    with warnings.catch_warnings():
        warnings.simplefilter("ignore")
        ref32 = c_ref.astype(np.float32).astype(np.float64)
    inf_r = np.isinf(ref32)
    inf_g = np.isinf(c)
    assert np.array_equal(inf_r, inf_g), f"{what}: inf positions differ"
    assert np.array_equal(c[inf_r], ref32[inf_r]), f"{what}: inf signs differ"
    fin = ~(nan_r | inf_r)
    tol = pam_ref.gemm_tolerance(s_ref[fin], k)
    err = np.abs(c[fin] - c_ref[fin])
    if err.size:
        worst = np.argmax(err / tol)
        assert np.all(err <= tol), (f"{what}: {int((err > tol).sum())} of {err.size} outputs outside tolerance; "
                                    f"worst err {err[worst]:.3e} vs tol {tol[worst]:.3e}")
