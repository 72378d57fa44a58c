"""Piecewise affine multiplication (PAM) on AMD Instinct MI355X (gfx950).

Thin Python binding over the C ABI in ``include/pam.h`` (libpam.so, built
from ``csrc/``).  The binding only marshals arguments: every step of the
computation runs in the library's HIP kernels, on the caller's current HIP
stream.  There is no CPU fallback; without the built library or a gfx950
device every call raises.

    mul(a, b, out=None)                        elementwise a .^ b
    pad(a, b, out=None)                        elementwise a ./ b (Sec. 2.3)
    palog2(a, out=None), paexp2(a, out=None)   elementwise (Sec. 2.3)
    round_mantissa(a, bits, out=None)          a rounded to `bits` mantissa bits
    gemm(A, B, trans_a, trans_b, out=None)     C = op(A) .^ op(B) (float32 or bfloat16 A, B)
    bmm(A, B, trans_a, trans_b, out=None)      batched over the leading axis
    exact_grad(A, B, Mod, trans_a, out=None)   exact-derivative product (Table 1)

Matrix arguments are float32 HIP tensors whose last dimension is contiguous
(row stride = leading dimension).  Products that split K take their
workspace from torch's caching allocator (the library's ``*_ws`` entry
points), so a call never waits for the GPU.  Every tensor of a call must be
on one device, which the call makes current.  op(X) = X^T when trans_x is
True.  The linear layer Y = X W^T is ``gemm(X, W, trans_b=True)``; its backward
products (approximate derivative, Table 1 of the paper) are
``gemm(dY, W)`` and ``gemm(dY, X, trans_a=True)``.
"""
from __future__ import annotations

import ctypes
import os

__all__ = ["mul", "pad", "palog2", "paexp2", "round_mantissa", "gemm", "bmm", "exact_grad", "plan",
           "device_info", "library_path", "load", "PamError"]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpam.so")

PAM_OP_N, PAM_OP_T = 0, 1


class PamError(RuntimeError):
    pass


class _Plan(ctypes.Structure):
    _fields_ = [("tile_m", ctypes.c_int32), ("tile_n", ctypes.c_int32), ("splits", ctypes.c_int32),
                ("kgroups", ctypes.c_int32), ("whole_tiles", ctypes.c_int64)]


class _DeviceInfo(ctypes.Structure):
    _fields_ = [("compute_units", ctypes.c_int32), ("simds_per_cu", ctypes.c_int32),
                ("lanes_per_simd", ctypes.c_int32), ("clock_khz", ctypes.c_int32),
                ("wavefront_size", ctypes.c_int32), ("valu_lane_ops_per_s", ctypes.c_double),
                ("arch", ctypes.c_char * 64)]


_lib = None

# Every symbol include/pam.h declares.
EXPORTS = ("pam_mul", "pam_pad", "pam_palog2", "pam_paexp2", "pam_round_mantissa", "pam_gemm", "pam_gemm_batched",
           "pam_gemm_narrow", "pam_gemm_exact_grad", "pam_gemm_plan", "pam_gemm_plan_for_workspace",
           "pam_gemm_batched_with_plan", "pam_gemm_plan_workspace_size", "pam_gemm_workspace_size",
           "pam_gemm_batched_ws", "pam_gemm_batched_noalloc", "pam_gemm_batched_bf16",
           "pam_gemm_exact_grad_workspace_size", "pam_gemm_exact_grad_ws", "pam_device_info", "pam_status_string",
           "pam_last_error")


def library_path() -> str:
    return LIB_PATH


def load() -> ctypes.CDLL:
    """Load libpam.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise PamError(f"{LIB_PATH} is missing: build it with `python -m paper_2305_17190_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    i64, vp, i32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
    lib.pam_mul.argtypes = [vp, vp, vp, i64, vp]
    lib.pam_pad.argtypes = [vp, vp, vp, i64, vp]
    lib.pam_palog2.argtypes = [vp, vp, i64, vp]
    lib.pam_paexp2.argtypes = [vp, vp, i64, vp]
    lib.pam_round_mantissa.argtypes = [vp, vp, i64, i32, vp]
    lib.pam_gemm_narrow.argtypes = [i32, i32, i64, i64, i64, vp, i64, i64, vp, i64, i64, vp, i64, i64, i64, i32, vp]
    lib.pam_gemm_exact_grad.argtypes = [i32, i64, i64, i64, vp, i64, vp, i64, vp, i64, vp, i64, vp]
    lib.pam_gemm.argtypes = [i32, i32, i64, i64, i64, vp, i64, vp, i64, vp, i64, vp]
    lib.pam_gemm_batched.argtypes = [i32, i32, i64, i64, i64, vp, i64, i64, vp, i64, i64, vp, i64, i64, i64, vp]
    sz, psz = ctypes.c_size_t, ctypes.POINTER(ctypes.c_size_t)
    lib.pam_gemm_batched_with_plan.argtypes = [i32, i32, i64, i64, i64, vp, i64, i64, vp, i64, i64, vp, i64, i64,
                                               i64, ctypes.POINTER(_Plan), vp, sz, vp]
    lib.pam_gemm_plan_workspace_size.argtypes = [i64, i64, i64, i64, ctypes.POINTER(_Plan), psz]
    lib.pam_gemm_plan.argtypes = [i64, i64, i64, i64, ctypes.POINTER(_Plan)]
    lib.pam_gemm_plan_for_workspace.argtypes = [i64, i64, i64, i64, ctypes.c_size_t, ctypes.POINTER(_Plan)]
    lib.pam_device_info.argtypes = [i32, ctypes.POINTER(_DeviceInfo)]
    lib.pam_gemm_workspace_size.argtypes = [i64, i64, i64, i64, psz]
    lib.pam_gemm_batched_ws.argtypes = [i32, i32, i64, i64, i64, vp, i64, i64, vp, i64, i64, vp, i64, i64, i64, i32,
                                        vp, sz, vp]
    lib.pam_gemm_batched_noalloc.argtypes = [i32, i32, i64, i64, i64, vp, i64, i64, vp, i64, i64, vp, i64, i64, i64,
                                             i32, vp]
    lib.pam_gemm_batched_bf16.argtypes = [i32, i32, i64, i64, i64, vp, i64, i64, vp, i64, i64, vp, i64, i64, i64,
                                          vp, sz, vp]
    lib.pam_gemm_exact_grad_workspace_size.argtypes = [i64, i64, i64, psz]
    lib.pam_gemm_exact_grad_ws.argtypes = [i32, i64, i64, i64, vp, i64, vp, i64, vp, i64, vp, i64, vp, sz, vp]
    for name in ("pam_mul", "pam_pad", "pam_palog2", "pam_paexp2", "pam_round_mantissa", "pam_gemm",
                 "pam_gemm_batched", "pam_gemm_narrow", "pam_gemm_exact_grad", "pam_gemm_batched_with_plan",
                 "pam_gemm_plan_workspace_size", "pam_gemm_plan", "pam_gemm_plan_for_workspace", "pam_device_info",
                 "pam_gemm_workspace_size", "pam_gemm_batched_ws", "pam_gemm_batched_noalloc",
                 "pam_gemm_batched_bf16",
                 "pam_gemm_exact_grad_workspace_size", "pam_gemm_exact_grad_ws"):
        getattr(lib, name).restype = i32
    lib.pam_status_string.argtypes = [i32]
    lib.pam_status_string.restype = ctypes.c_char_p
    lib.pam_last_error.argtypes = []
    lib.pam_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != 0:
        lib = load()
        raise PamError(f"{lib.pam_status_string(status).decode()}: {lib.pam_last_error().decode()}")


def _torch():
    import torch
    return torch


def _stream_handle(t) -> int:
    torch = _torch()
    return torch.cuda.current_stream(t.device).cuda_stream


# Split-K workspace bytes per (kind, sizes), as the library reports them.
_ws_bytes = {}


def _workspace(kind: str, sizes: tuple, device):
    """(pointer, bytes, tensor) of the split-K workspace a product needs, taken
    from torch's caching allocator on the current stream (stream-ordered, so
    it stays reserved until the product's kernels are done); (None, 0, None)
    when the product does not split K."""
    key = (kind,) + sizes
    nbytes = _ws_bytes.get(key)
    if nbytes is None:
        out = ctypes.c_size_t()
        fn = load().pam_gemm_workspace_size if kind == "gemm" else load().pam_gemm_exact_grad_workspace_size
        _check(fn(*sizes, ctypes.byref(out)))
        nbytes = int(out.value)
        if len(_ws_bytes) >= 4096:
            _ws_bytes.clear()
        _ws_bytes[key] = nbytes
    if nbytes == 0:
        return None, 0, None
    buf = _torch().empty(nbytes, dtype=_torch().uint8, device=device)
    return buf.data_ptr(), nbytes, buf


def _require(t, name: str, ndim: int, bf16_ok: bool = False):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != torch.float32 and not (bf16_ok and t.dtype == torch.bfloat16):
        raise TypeError(f"{name} must be float32{' or bfloat16' if bf16_ok else ''}, got {t.dtype}")
    if not t.is_cuda:
        raise PamError(f"{name} must be a HIP (cuda) tensor; the PAM library has no CPU path")
    if t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions, got {t.dim()}")
    if t.numel() > 0 and t.stride(-1) != 1:
        raise ValueError(f"{name} must have a contiguous last dimension")


def _same_device(ref, *named):
    """The library launches on the current HIP device: every tensor of a call
    must live on the first operand's device (made current for the call)."""
    for name, t in named:
        if t is not None and t.device != ref.device:
            raise ValueError(f"{name} is on {t.device}, the first operand on {ref.device}")


def _elementwise_args(tensors, out):
    torch = _torch()
    for name, t in tensors:
        _require(t, name, t.dim() if isinstance(t, torch.Tensor) else 1)
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    a = tensors[0][1]
    _same_device(a, *tensors[1:])
    for name, t in tensors[1:]:
        if t.shape != a.shape:
            raise ValueError(f"shape mismatch {tuple(a.shape)} vs {tuple(t.shape)}")
    if out is None:
        out = torch.empty_like(a)
    elif (not isinstance(out, torch.Tensor) or out.shape != a.shape or not out.is_contiguous()
          or out.dtype != torch.float32 or out.device != a.device):
        raise ValueError("out must be a contiguous float32 tensor of the same shape and device")
    return a, out


def mul(a, b, out=None):
    """Elementwise PAM of two equally shaped contiguous float32 tensors."""
    a, out = _elementwise_args((("a", a), ("b", b)), out)
    with _torch().cuda.device(a.device):
        _check(load().pam_mul(a.data_ptr(), b.data_ptr(), out.data_ptr(), a.numel(), _stream_handle(a)))
    return out


def pad(a, b, out=None):
    """Elementwise piecewise affine division a ./ b (Sec. 2.3)."""
    a, out = _elementwise_args((("a", a), ("b", b)), out)
    with _torch().cuda.device(a.device):
        _check(load().pam_pad(a.data_ptr(), b.data_ptr(), out.data_ptr(), a.numel(), _stream_handle(a)))
    return out


def palog2(a, out=None):
    """Elementwise palog2(a) = E + M (Sec. 2.3), rounded to float32."""
    a, out = _elementwise_args((("a", a),), out)
    with _torch().cuda.device(a.device):
        _check(load().pam_palog2(a.data_ptr(), out.data_ptr(), a.numel(), _stream_handle(a)))
    return out


def paexp2(a, out=None):
    """Elementwise paexp2(a) = 2^floor(a) (1 + a - floor(a)) (Sec. 2.3), rounded to float32."""
    a, out = _elementwise_args((("a", a),), out)
    with _torch().cuda.device(a.device):
        _check(load().pam_paexp2(a.data_ptr(), out.data_ptr(), a.numel(), _stream_handle(a)))
    return out


def round_mantissa(a, bits: int, out=None):
    """Elementwise rounding to ``bits`` mantissa bits (App. "PAM with Narrower Mantissas")."""
    a, out = _elementwise_args((("a", a),), out)
    with _torch().cuda.device(a.device):
        _check(load().pam_round_mantissa(a.data_ptr(), out.data_ptr(), a.numel(), int(bits), _stream_handle(a)))
    return out


def _bf16_pair(A, B, mantissa_bits) -> bool:
    """True for two bfloat16 operands (their values already have 7 mantissa
    bits); mixed float32 / bfloat16 operands are refused."""
    torch = _torch()
    a16, b16 = A.dtype == torch.bfloat16, B.dtype == torch.bfloat16
    if a16 != b16:
        raise TypeError("A and B must both be float32 or both bfloat16")
    if a16 and int(mantissa_bits) < 7:
        raise ValueError("bfloat16 operands have 7 mantissa bits; round float32 operands for fewer")
    return a16


def _dims(A, B, trans_a: bool, trans_b: bool):
    m, k = (A.shape[-1], A.shape[-2]) if trans_a else (A.shape[-2], A.shape[-1])
    kb, n = (B.shape[-1], B.shape[-2]) if trans_b else (B.shape[-2], B.shape[-1])
    if k != kb:
        raise ValueError(f"inner dimensions differ: op(A) is {m}x{k}, op(B) is {kb}x{n}")
    return m, n, k


def _ld(t) -> int:
    return max(int(t.stride(-2)), 1) if t.numel() > 0 else max(int(t.shape[-1]), 1)


def gemm(A, B, trans_a: bool = False, trans_b: bool = False, out=None, mantissa_bits: int = 23):
    """C = op(A) .^ op(B) with float32 accumulation; returns C (m x n).

    ``mantissa_bits`` < 23 rounds every operand element to that many mantissa
    bits first (App. "PAM with Narrower Mantissas").  A and B may both be
    bfloat16 (7-bit mantissas in half the bytes): the kernels widen them
    exactly to float32 as they load them; C is float32."""
    torch = _torch()
    _require(A, "A", 2, bf16_ok=True)
    _require(B, "B", 2, bf16_ok=True)
    bf16 = _bf16_pair(A, B, mantissa_bits)
    m, n, k = _dims(A, B, trans_a, trans_b)
    if out is None:
        out = torch.empty((m, n), dtype=torch.float32, device=A.device)
    else:
        _require(out, "out", 2)
        if tuple(out.shape) != (m, n):
            raise ValueError(f"out must be {m}x{n}")
    _same_device(A, ("B", B), ("out", out))
    ta = PAM_OP_T if trans_a else PAM_OP_N
    tb = PAM_OP_T if trans_b else PAM_OP_N
    lib = load()
    with torch.cuda.device(A.device):
        ws, ws_bytes, keep = _workspace("gemm", (m, n, k, 1), A.device)
        if bf16:
            _check(lib.pam_gemm_batched_bf16(ta, tb, m, n, k, A.data_ptr(), _ld(A), 0, B.data_ptr(), _ld(B), 0,
                                             out.data_ptr(), _ld(out), 0, 1, ws, ws_bytes, _stream_handle(A)))
        else:
            _check(lib.pam_gemm_batched_ws(ta, tb, m, n, k, A.data_ptr(), _ld(A), 0, B.data_ptr(), _ld(B), 0,
                                           out.data_ptr(), _ld(out), 0, 1, int(mantissa_bits), ws, ws_bytes,
                                           _stream_handle(A)))
        del keep
    return out


def bmm(A, B, trans_a: bool = False, trans_b: bool = False, out=None, plan=None, mantissa_bits: int = 23):
    """Batched C[z] = op(A[z]) .^ op(B[z]) over the leading axis.

    ``plan`` = (tile_m, tile_n, splits[, kgroups[, whole_tiles]]) forces a
    tiling (tests and tuning); ``whole_tiles`` tiles, counted from the first,
    then take the whole K and only the rest are split.  ``mantissa_bits`` <
    23 rounds every operand element to that many mantissa bits first (the
    library then picks the plan).
    """
    torch = _torch()
    _require(A, "A", 3, bf16_ok=True)
    _require(B, "B", 3, bf16_ok=True)
    bf16 = _bf16_pair(A, B, mantissa_bits)
    if A.shape[0] != B.shape[0]:
        raise ValueError("batch sizes differ")
    batch = A.shape[0]
    m, n, k = _dims(A, B, trans_a, trans_b)
    if out is None:
        out = torch.empty((batch, m, n), dtype=torch.float32, device=A.device)
    else:
        _require(out, "out", 3)
        if tuple(out.shape) != (batch, m, n):
            raise ValueError(f"out must be {batch}x{m}x{n}")
    _same_device(A, ("B", B), ("out", out))
    ta = PAM_OP_T if trans_a else PAM_OP_N
    tb = PAM_OP_T if trans_b else PAM_OP_N
    args = (ta, tb, m, n, k, A.data_ptr(), _ld(A), A.stride(0), B.data_ptr(), _ld(B), B.stride(0),
            out.data_ptr(), _ld(out), out.stride(0), batch)
    if bf16 and plan is not None:
        raise ValueError("bfloat16 operands take the library's plan")
    if plan is not None and mantissa_bits != 23:
        raise ValueError("plan and mantissa_bits cannot be combined")
    if plan is not None and not 3 <= len(plan) <= 5:
        raise ValueError("plan is (tile_m, tile_n, splits[, kgroups[, whole_tiles]])")
    lib = load()
    with torch.cuda.device(A.device):
        if plan is not None:
            full = tuple(plan) + (1, 0)[len(plan) - 3:]
            p = _Plan(*full)
            need = ctypes.c_size_t()
            _check(lib.pam_gemm_plan_workspace_size(m, n, k, batch, ctypes.byref(p), ctypes.byref(need)))
            keep = torch.empty(int(need.value), dtype=torch.uint8, device=A.device) if need.value else None
            _check(lib.pam_gemm_batched_with_plan(*args, ctypes.byref(p), keep.data_ptr() if keep is not None else None,
                                                  int(need.value), _stream_handle(A)))
            del keep
            return out
        ws, ws_bytes, keep = _workspace("gemm", (m, n, k, batch), A.device)
        if bf16:
            _check(lib.pam_gemm_batched_bf16(*args, ws, ws_bytes, _stream_handle(A)))
        else:
            _check(lib.pam_gemm_batched_ws(*args, int(mantissa_bits), ws, ws_bytes, _stream_handle(A)))
        del keep
    return out


def exact_grad(A, B, Mod, trans_a: bool = False, out=None):
    """C(r, c) = sum_q op(A)(r, q) d(Mod(r, c) .^ B(q, c)) / dMod(r, c) (Table 1's
    exact derivative: zero where Mod .^ B is clamped).  For Y = X .^ W^T: dX = exact_grad(dY, W, X) and
    dW = exact_grad(dY, X, W, trans_a=True)."""
    torch = _torch()
    _require(A, "A", 2)
    _require(B, "B", 2)
    _require(Mod, "Mod", 2)
    m, k = (A.shape[1], A.shape[0]) if trans_a else (A.shape[0], A.shape[1])
    if B.shape[0] != k:
        raise ValueError(f"inner dimensions differ: op(A) is {m}x{k}, B is {tuple(B.shape)}")
    n = B.shape[1]
    if tuple(Mod.shape) != (m, n):
        raise ValueError(f"Mod must be {m}x{n}")
    if out is None:
        out = torch.empty((m, n), dtype=torch.float32, device=A.device)
    else:
        _require(out, "out", 2)
        if tuple(out.shape) != (m, n):
            raise ValueError(f"out must be {m}x{n}")
    _same_device(A, ("B", B), ("Mod", Mod), ("out", out))
    with torch.cuda.device(A.device):
        ws, ws_bytes, keep = _workspace("exact", (m, n, k), A.device)
        _check(load().pam_gemm_exact_grad_ws(PAM_OP_T if trans_a else PAM_OP_N, m, n, k, A.data_ptr(), _ld(A),
                                             B.data_ptr(), _ld(B), Mod.data_ptr(), _ld(Mod), out.data_ptr(),
                                             _ld(out), ws, ws_bytes, _stream_handle(A)))
        del keep
    return out


def plan(m: int, n: int, k: int, batch: int = 1, max_workspace_bytes: int | None = None):
    """(tile_m, tile_n, splits, kgroups, whole_tiles) the library picks for
    these sizes: with no limit (the plan gemm / bmm use, their split-K
    workspace taken from torch), or the fastest whose split-K partial sums
    fit in ``max_workspace_bytes`` (0: the C entry points without a
    workspace argument)."""
    p = _Plan()
    if max_workspace_bytes is None:
        _check(load().pam_gemm_plan(m, n, k, batch, ctypes.byref(p)))
    else:
        _check(load().pam_gemm_plan_for_workspace(m, n, k, batch, int(max_workspace_bytes), ctypes.byref(p)))
    return (p.tile_m, p.tile_n, p.splits, p.kgroups, p.whole_tiles)


def device_info(device: int = 0) -> dict:
    info = _DeviceInfo()
    _check(load().pam_device_info(device, ctypes.byref(info)))
    return {"compute_units": info.compute_units, "simds_per_cu": info.simds_per_cu,
            "lanes_per_simd": info.lanes_per_simd, "clock_khz": info.clock_khz,
            "wavefront_size": info.wavefront_size, "valu_lane_ops_per_s": info.valu_lane_ops_per_s,
            "arch": info.arch.decode()}
