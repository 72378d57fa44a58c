"""Seeded synthetic inputs for the PAM GEMM workloads.

This module only draws numbers and describes shapes.  It holds none of the
arithmetic of piecewise affine multiplication, so both the CPU oracle and the
HIP path can take their inputs from it without sharing any method code.

Every tensor is generated on the CPU in float32 with numpy's PCG64 generator
seeded with ``1000 * workload + tensor_id``, so the oracle and the GPU see the
same bits.  The shapes and distributions stand in for the paper's workloads
(the DeiT-Tiny vision transformer and the IWSLT14 encoder-decoder transformer
of Sec. 3.1, whose datasets and weights are not used here):

  w1  single 256^3 GEMM, N(0,1) operands; plus a 2^20-element elementwise
      input pair with 1% exact zeros and 1% signed powers of two
  w2  ViT-tiny linear layer: X[64*197=12608, 192] ~ N(0,1),
      W[768, 192] ~ N(0, 0.02^2), dY[12608, 768] ~ N(0, 1e-3^2)
  w3  transformer-base FFN: tokens 8192, d_model 512, d_ff 2048; X, H, dZ, dH
      ~ N(0,1); W1[2048, 512], W2[512, 2048] ~ Xavier-uniform
  w4  batched attention: 32 x 8 heads, seq 256, head dim 64; Q, K, V, dO
      ~ N(0,1); P = row softmax of N(0,1) logits; dS ~ N(0,1)
  w5  large linear: X[16384, 4096] ~ N(0,1), W[4096, 4096] ~ N(0, 1/4096),
      dY[16384, 4096] ~ N(0, 1e-4^2); in each tensor 0.1% of the entries are
      exact signed zeros and 0.1% are +-u * 2^-126 with u ~ U[0.5, 2)
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

MIN_NORMAL_F32 = float(np.finfo(np.float32).tiny)  # 2^-126


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def normal(shape, std: float, seed: int) -> np.ndarray:
    z = rng(seed).standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        z *= np.float32(std)
    return z


def uniform(shape, bound: float, seed: int) -> np.ndarray:
    return rng(seed).uniform(-bound, bound, size=shape).astype(np.float32)


def inject_zeros_and_tiny(x: np.ndarray, frac_zero: float, frac_tiny: float, seed: int) -> np.ndarray:
    """Overwrite random entries with signed zeros and values near 2^-126.

    Half of the tiny values (u < 1) are denormal inputs, the other half are
    small normals whose products underflow.
    """
    g = rng(seed)
    flat = x.reshape(-1)
    n = flat.size
    nz = int(round(n * frac_zero))
    nt = int(round(n * frac_tiny))
    idx = g.choice(n, size=nz + nt, replace=False) if n < (1 << 22) else g.integers(0, n, size=nz + nt)
    zsign = np.where(g.random(nz) < 0.5, np.float32(0.0), np.float32(-0.0)).astype(np.float32)
    flat[idx[:nz]] = zsign
    u = g.uniform(0.5, 2.0, size=nt)
    sgn = np.where(g.random(nt) < 0.5, 1.0, -1.0)
    flat[idx[nz:]] = (sgn * u * MIN_NORMAL_F32).astype(np.float32)
    return x


def exact_sum_values(shape, seed: int, frac_zero: float = 0.001, frac_tiny: float = 0.001) -> np.ndarray:
    """float32 values with two mantissa bits and exponents in [-6, -3]:
    (-1)^s 2^e (1 + j/4).  Any sum of products of such values (PAM or true
    products: both are multiples of 2^-14 below 2^-4) stays exact in float32
    for up to 2^16 terms, in every summation order.  Planted: signed zeros,
    denormals, and tiny normals (+-u 2^-126, u in [1, 4)) that vanish in every
    such product, so the exact-sum property holds while the zero and tiny
    values still appear in the operands.
    """
    g = rng(seed)
    e = g.integers(-6, -2, size=shape)
    j = g.integers(0, 4, size=shape)
    sgn = np.where(g.random(shape) < 0.5, -1.0, 1.0)
    x = (sgn * np.ldexp(1.0 + j / 4.0, e)).astype(np.float32)
    u = g.random(shape)
    tiny = (sgn * g.uniform(1.0, 4.0, size=shape) * MIN_NORMAL_F32).astype(np.float32)
    denorm = (sgn * g.uniform(0.01, 0.99, size=shape) * MIN_NORMAL_F32).astype(np.float32)
    zero = np.where(sgn < 0, np.float32(-0.0), np.float32(0.0)).astype(np.float32)
    x = np.where(u < frac_zero, zero, x)
    x = np.where((u >= frac_zero) & (u < frac_zero + frac_tiny / 2), denorm, x)
    x = np.where((u >= frac_zero + frac_tiny / 2) & (u < frac_zero + frac_tiny), tiny, x)
    return x.astype(np.float32)


def row_softmax(logits: np.ndarray) -> np.ndarray:
    """Ordinary float32 softmax along the last axis (data generation only)."""
    m = logits.max(axis=-1, keepdims=True)
    e = np.exp(logits - m, dtype=np.float32)
    return (e / e.sum(axis=-1, keepdims=True, dtype=np.float32)).astype(np.float32)


# ---------------------------------------------------------------------------
# Elementwise inputs
# ---------------------------------------------------------------------------

def pam_mul_inputs(n: int, seed: int) -> Tuple[np.ndarray, np.ndarray]:
    """a, b ~ N(0,1); 1% of each set to signed zeros, 1% to +-2^k, k in [-20, 20]."""
    g = rng(seed)
    out = []
    for _ in range(2):
        x = g.standard_normal(size=n, dtype=np.float32)
        m = max(1, n // 100) if n >= 100 else 0
        if m:
            idx = g.choice(n, size=2 * m, replace=False)
            x[idx[:m]] = np.where(g.random(m) < 0.5, 0.0, -0.0).astype(np.float32)
            k = g.integers(-20, 21, size=m)
            s = np.where(g.random(m) < 0.5, 1.0, -1.0)
            x[idx[m:]] = (s * np.ldexp(1.0, k)).astype(np.float32)
        out.append(x)
    return out[0], out[1]


def paexp2_arguments(n: int, seed: int) -> np.ndarray:
    """Arguments of paexp2 as piecewise affine softmax and exp produce them:
    half x - max(x) of N(0, 4^2) logits (mostly in [-30, 0]), a quarter
    U(-140, 140) (both saturations), a quarter small |x| < 1 of random
    exponents (where the result needs rounding)."""
    g = rng(seed)
    h, q = n // 2, n // 4
    logits = (4.0 * g.standard_normal(size=h)).astype(np.float32)
    a = (logits - logits.max()).astype(np.float32) if h else logits
    b = g.uniform(-140.0, 140.0, size=q).astype(np.float32)
    c_bits = ((g.integers(0, 2, size=n - h - q) << 31) | (g.integers(60, 127, size=n - h - q) << 23)
              | g.integers(0, 1 << 23, size=n - h - q)).astype(np.uint32)
    x = np.concatenate([a, b, c_bits.view(np.float32)])
    return x[g.permutation(n)]


def random_bit_patterns(n: int, seed: int) -> np.ndarray:
    """Uniformly random 32-bit patterns viewed as float32 (all classes)."""
    return rng(seed).integers(0, 1 << 32, size=n, dtype=np.uint64).astype(np.uint32).view(np.float32)


def special_bit_patterns() -> np.ndarray:
    """Edge-case float32 encodings: zeros, denormals, boundaries, specials."""
    pos = [
        0x00000000,  # +0
        0x00000001,  # smallest denormal
        0x007FFFFF,  # largest denormal
        0x00400000,  # mid denormal
        0x00800000,  # min normal 2^-126
        0x00800001,
        0x00C00000,  # 1.5 * 2^-126
        0x1F800000,  # 2^-64
        0x1FC00000,  # 1.5 * 2^-64
        0x1FA00000,  # 1.25 * 2^-64
        0x20000000,  # 2^-63
        0x20400000,  # 1.5 * 2^-63
        0x20200000,  # 1.25 * 2^-63
        0x3F000000,  # 0.5
        0x3F800000,  # 1
        0x3F800001,  # 1 + ulp
        0x3FC00000,  # 1.5
        0x3FFFFFFF,  # just below 2
        0x40000000,  # 2
        0x40400000,  # 3
        0x5F800000,  # 2^64
        0x5F7FFFFF,  # just below 2^64
        0x5FC00000,  # 1.5 * 2^64
        0x7F000000,  # 2^127
        0x7F7FFFFF,  # FLT_MAX
        0x7F800000,  # +inf
        0x7FC00000,  # quiet NaN
        0x7F800001,  # signalling NaN
        0x7FFFFFFF,  # NaN, all payload bits
    ]
    allbits = pos + [p | 0x80000000 for p in pos]
    return np.array(allbits, dtype=np.uint32).view(np.float32)


# ---------------------------------------------------------------------------
# GEMM workloads
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class GemmForm:
    """One product C = op(A) .^ op(B) of a workload, row-major operands.

    op(A) is M x K: A[i*lda + k] when trans_a is False, A[k*lda + i] when True.
    op(B) is K x N: B[k*ldb + j] when trans_b is False, B[j*ldb + k] when True.
    """
    name: str
    a: str
    b: str
    trans_a: bool
    trans_b: bool
    m: int
    n: int
    k: int
    lda: int
    ldb: int
    ldc: int
    batch: int = 1
    stride_a: int = 0
    stride_b: int = 0
    stride_c: int = 0

    @property
    def macs(self) -> int:
        return self.m * self.n * self.k * self.batch

    @property
    def min_bytes(self) -> int:
        return 4 * (self.m * self.k + self.k * self.n + self.m * self.n) * self.batch


def _lin(name, a, b, ta, tb, m, n, k, lda, ldb):
    return GemmForm(name, a, b, ta, tb, m, n, k, lda, ldb, n)


def _bmm(name, a, b, ta, tb, m, n, k, lda, ldb, sa, sb, batch):
    return GemmForm(name, a, b, ta, tb, m, n, k, lda, ldb, n, batch, sa, sb, m * n)


WORKLOADS: Dict[int, dict] = {
    1: dict(
        name="w1_gemm256",
        desc="single PAM GEMM 256x256x256, N(0,1) operands",
        forms=[
            _lin("nn", "A", "B", False, False, 256, 256, 256, 256, 256),
            _lin("nt", "A", "B", False, True, 256, 256, 256, 256, 256),
            _lin("tn", "A", "B", True, False, 256, 256, 256, 256, 256),
            _lin("tt", "A", "B", True, True, 256, 256, 256, 256, 256),
        ],
    ),
    2: dict(
        name="w2_vit_tiny_linear",
        desc="ViT-tiny linear 12608x192 -> 768: fwd, dX, dW",
        forms=[
            _lin("fwd", "X", "W", False, True, 12608, 768, 192, 192, 192),
            _lin("dX", "dY", "W", False, False, 12608, 192, 768, 768, 192),
            _lin("dW", "dY", "X", True, False, 768, 192, 12608, 768, 192),
        ],
    ),
    3: dict(
        name="w3_transformer_base_ffn",
        desc="transformer-base FFN, 8192 tokens, 512 -> 2048 -> 512: up, down and their dX, dW",
        forms=[
            _lin("up", "X", "W1", False, True, 8192, 2048, 512, 512, 512),
            _lin("down", "H", "W2", False, True, 8192, 512, 2048, 2048, 2048),
            _lin("dH", "dZ", "W2", False, False, 8192, 2048, 512, 512, 2048),
            _lin("dW2", "dZ", "H", True, False, 512, 2048, 8192, 512, 2048),
            _lin("dX", "dH", "W1", False, False, 8192, 512, 2048, 2048, 512),
            _lin("dW1", "dH", "X", True, False, 2048, 512, 8192, 2048, 512),
        ],
    ),
    4: dict(
        name="w4_attention_bmm",
        desc="batched attention 256 x (256x256, head 64): QK^T, PV and their backward products",
        forms=[
            _bmm("QKt", "Q", "K", False, True, 256, 256, 64, 64, 64, 16384, 16384, 256),
            _bmm("PV", "P", "V", False, False, 256, 64, 256, 256, 64, 65536, 16384, 256),
            _bmm("dP", "dO", "V", False, True, 256, 256, 64, 64, 64, 16384, 16384, 256),
            _bmm("dV", "P", "dO", True, False, 256, 64, 256, 256, 64, 65536, 16384, 256),
            _bmm("dQ", "dS", "K", False, False, 256, 64, 256, 256, 64, 65536, 16384, 256),
            _bmm("dK", "dS", "Q", True, False, 256, 64, 256, 256, 64, 65536, 16384, 256),
        ],
    ),
    5: dict(
        name="w5_large_linear",
        desc="large linear 16384 tokens, 4096 -> 4096: fwd, dX, dW, with zeros and near-min-normal values",
        forms=[
            _lin("fwd", "X", "W", False, True, 16384, 4096, 4096, 4096, 4096),
            _lin("dX", "dY", "W", False, False, 16384, 4096, 4096, 4096, 4096),
            _lin("dW", "dY", "X", True, False, 4096, 4096, 16384, 4096, 4096),
        ],
    ),
}


def workload_inputs(w: int, only: Optional[List[str]] = None) -> Dict[str, np.ndarray]:
    """All input tensors of workload ``w`` (float32, row-major, contiguous)."""
    s = 1000 * w
    want = (lambda name: only is None or name in only)
    t: Dict[str, np.ndarray] = {}
    if w == 1:
        if want("A"):
            t["A"] = normal((256, 256), 1.0, s + 1)
        if want("B"):
            t["B"] = normal((256, 256), 1.0, s + 2)
    elif w == 2:
        if want("X"):
            t["X"] = normal((12608, 192), 1.0, s + 1)
        if want("W"):
            t["W"] = normal((768, 192), 0.02, s + 2)
        if want("dY"):
            t["dY"] = normal((12608, 768), 1e-3, s + 3)
    elif w == 3:
        bound = float(np.sqrt(6.0 / (512 + 2048)))
        if want("X"):
            t["X"] = normal((8192, 512), 1.0, s + 1)
        if want("H"):
            t["H"] = normal((8192, 2048), 1.0, s + 2)
        if want("dZ"):
            t["dZ"] = normal((8192, 512), 1.0, s + 3)
        if want("dH"):
            t["dH"] = normal((8192, 2048), 1.0, s + 4)
        if want("W1"):
            t["W1"] = uniform((2048, 512), bound, s + 5)
        if want("W2"):
            t["W2"] = uniform((512, 2048), bound, s + 6)
    elif w == 4:
        for i, name in enumerate(["Q", "K", "V", "dO"]):
            if want(name):
                t[name] = normal((256, 256, 64), 1.0, s + 1 + i)
        if want("P"):
            t["P"] = row_softmax(normal((256, 256, 256), 1.0, s + 5))
        if want("dS"):
            t["dS"] = normal((256, 256, 256), 1.0, s + 6)
    elif w == 5:
        if want("X"):
            t["X"] = inject_zeros_and_tiny(normal((16384, 4096), 1.0, s + 1), 1e-3, 1e-3, s + 11)
        if want("W"):
            t["W"] = inject_zeros_and_tiny(normal((4096, 4096), 1.0 / 64.0, s + 2), 1e-3, 1e-3, s + 12)
        if want("dY"):
            t["dY"] = inject_zeros_and_tiny(normal((16384, 4096), 1e-4, s + 3), 1e-3, 1e-3, s + 13)
    else:
        raise ValueError(f"unknown workload {w}")
    return t


def random_matrix(rows: int, cols: int, seed: int, std: float = 1.0) -> np.ndarray:
    return normal((rows, cols), std, seed)
