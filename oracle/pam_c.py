"""ctypes front end and build step for the plain C oracle (pam_oracle.c).

TEST INFRASTRUCTURE ONLY (tests, smoke check, benchmark CPU baseline).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "pam_oracle.c")
LIB = os.path.join(HERE, "libpam_oracle.so")

_lib = None


def build(verbose: bool = False) -> str:
    """Compile the C oracle with gcc -O2 (no fast-math) and OpenMP.  The
    library is written under a per-process name and renamed into place, so
    concurrent builds (parallel test workers) never see a partial file."""
    tmp = f"{LIB}.{os.getpid()}.tmp"
    cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-o", tmp, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def load() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB):
        build()
    lib = ctypes.CDLL(LIB)
    lib.pam_oracle_bits.restype = ctypes.c_uint32
    lib.pam_oracle_bits.argtypes = [ctypes.c_uint32, ctypes.c_uint32]
    lib.pam_oracle_mul.restype = None
    lib.pam_oracle_mul.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
    i64 = ctypes.c_int64
    lib.pam_oracle_gemm.restype = None
    lib.pam_oracle_gemm.argtypes = [ctypes.c_int, ctypes.c_int, i64,
                                    ctypes.c_void_p, i64, i64,
                                    ctypes.c_void_p, i64, i64,
                                    ctypes.c_void_p, i64,
                                    ctypes.c_void_p, i64,
                                    ctypes.c_void_p, i64,
                                    ctypes.c_void_p, ctypes.c_void_p]
    lib.pam_oracle_num_threads.restype = ctypes.c_int
    lib.pam_oracle_set_threads.restype = None
    lib.pam_oracle_set_threads.argtypes = [ctypes.c_int]
    _lib = lib
    return lib


def num_threads() -> int:
    return int(load().pam_oracle_num_threads())


def set_threads(n: int) -> None:
    """Thread count of the oracle's parallel loops from now on."""
    load().pam_oracle_set_threads(int(n))


def pam_mul(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32).reshape(-1)
    b = np.ascontiguousarray(b, dtype=np.float32).reshape(-1)
    out = np.empty_like(a)
    load().pam_oracle_mul(a.ctypes.data, b.ctypes.data, out.ctypes.data, a.size)
    return out


def _ptr(x: np.ndarray) -> int:
    return x.ctypes.data


def pam_gemm(a: np.ndarray, b: np.ndarray, trans_a: bool, trans_b: bool, m: int, n: int, k: int,
             lda: int, ldb: int, stride_a: int = 0, stride_b: int = 0,
             batches: Optional[Sequence[int]] = None,
             rows: Optional[Sequence[int]] = None,
             cols: Optional[Sequence[int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Sub-grid [len(batches), len(rows), len(cols)] of C and S = sum |term|.

    ``a`` and ``b`` are flat float32 buffers laid out with the given leading
    dimensions and batch strides (row-major, as the HIP library takes them).
    """
    a = np.ascontiguousarray(a, dtype=np.float32).reshape(-1)
    b = np.ascontiguousarray(b, dtype=np.float32).reshape(-1)
    bt = np.asarray([0] if batches is None else batches, dtype=np.int64)
    rt = np.asarray(np.arange(m) if rows is None else rows, dtype=np.int64)
    ct = np.asarray(np.arange(n) if cols is None else cols, dtype=np.int64)
    c = np.empty((bt.size, rt.size, ct.size), dtype=np.float64)
    s = np.empty_like(c)
    load().pam_oracle_gemm(int(trans_a), int(trans_b), k,
                           _ptr(a), lda, stride_a, _ptr(b), ldb, stride_b,
                           _ptr(bt), bt.size, _ptr(rt), rt.size, _ptr(ct), ct.size,
                           _ptr(c), _ptr(s))
    return c, s
