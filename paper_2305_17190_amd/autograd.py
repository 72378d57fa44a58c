"""PyTorch autograd wrappers over the PAM matrix products.

Sec. 3.2 of the paper replaces every multiplication of a linear layer and of
the attention's batched products by PAM, and Table 1 gives the backward pass
used in training, the approximate derivative: the gradients are PAM products
of the incoming gradient with the other operand, exactly as a standard
matrix multiply's gradients are ordinary products.

    Y = X .^ W^T (+ b)     dX = dY .^ W       dW = dY^T .^ X     db = sum dY
    C = A .^ B (batched)   dA = dC .^ B^T     dB = A^T .^ dC

Every product runs in the library's HIP kernels (``pam.gemm`` / ``pam.bmm``);
the bias gradient is an ordinary sum (no multiplication).  ``pam_linear``
and ``PAMLinear`` also offer Table 1's exact derivative
(``derivative="exact"``): dX[i,k] = sum_j dY[i,j] d(X[i,k] .^ W[j,k])/dX[i,k]
and dW likewise, through ``pam.exact_grad``.  With
``mantissa_bits`` < 23 every product, forward and backward, first rounds its
two operands to that many mantissa bits (App. "PAM with Narrower
Mantissas"); the tensors themselves are not modified.  Inputs must be float32
HIP tensors; there is no CPU path.
"""
from __future__ import annotations

import math

import torch

from . import bmm as _bmm
from . import exact_grad as _exact_grad
from . import gemm as _gemm

__all__ = ["pam_linear", "pam_matmul", "PAMLinear"]


def _float32(**named) -> None:
    """The wrappers' gradients are float32 products: refuse other dtypes up
    front rather than in the backward pass."""
    for name, t in named.items():
        if t is not None and t.dtype != torch.float32:
            raise TypeError(f"{name} must be float32, got {t.dtype}")


def _last_contiguous(t: torch.Tensor) -> torch.Tensor:
    """t itself when its rows are dense and non-overlapping (a valid leading
    dimension for the C ABI), else a contiguous copy."""
    ok = t.stride(-1) == 1 and (t.dim() < 2 or t.shape[-2] <= 1 or t.stride(-2) >= t.shape[-1])
    return t if ok else t.contiguous()


class _PAMLinearFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x2d, weight, bias, bits, exact):
        x2d = _last_contiguous(x2d)
        weight = _last_contiguous(weight)
        ctx.save_for_backward(x2d, weight)
        ctx.has_bias = bias is not None
        ctx.bits = bits
        ctx.exact = exact
        y = _gemm(x2d, weight, trans_b=True, mantissa_bits=bits)   # Y = X .^ W^T
        if bias is not None:
            y += bias
        return y

    @staticmethod
    def backward(ctx, dy):
        x2d, weight = ctx.saved_tensors
        dy = _last_contiguous(dy)
        dx = dw = db = None
        if ctx.exact:
            if ctx.needs_input_grad[0]:
                dx = _exact_grad(dy, weight, x2d)                           # sum_j dY d(X .^ W)/dX
            if ctx.needs_input_grad[1]:
                dw = _exact_grad(dy, x2d, weight, trans_a=True)             # sum_i dY d(W .^ X)/dW
        else:
            if ctx.needs_input_grad[0]:
                dx = _gemm(dy, weight, mantissa_bits=ctx.bits)              # dX = dY .^ W
            if ctx.needs_input_grad[1]:
                dw = _gemm(dy, x2d, trans_a=True, mantissa_bits=ctx.bits)   # dW = dY^T .^ X
        if ctx.has_bias and ctx.needs_input_grad[2]:
            db = dy.sum(dim=0)
        return dx, dw, db, None, None


def pam_linear(x: torch.Tensor, weight: torch.Tensor, bias: torch.Tensor = None,
               mantissa_bits: int = 23, derivative: str = "approximate") -> torch.Tensor:
    """``x .^ weight^T + bias`` over the last dimension of x (any leading dims).

    ``derivative``: "approximate" (Table 1's approximate derivative, PAM
    products) or "exact" (Table 1's exact derivative)."""
    if x.dim() < 1:
        raise ValueError("x must have at least one dimension")
    if derivative not in ("approximate", "exact"):
        raise ValueError('derivative must be "approximate" or "exact"')
    if derivative == "exact" and mantissa_bits != 23:
        raise ValueError("the exact derivative takes full float32 mantissas")
    _float32(x=x, weight=weight, bias=bias)
    lead = x.shape[:-1]
    y = _PAMLinearFn.apply(x.reshape(-1, x.shape[-1]), weight, bias, int(mantissa_bits), derivative == "exact")
    return y.reshape(*lead, weight.shape[0])


class _PAMBmmFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, a, b, bits):
        a = _last_contiguous(a)
        b = _last_contiguous(b)
        ctx.save_for_backward(a, b)
        ctx.bits = bits
        return _bmm(a, b, mantissa_bits=bits)                 # C = A .^ B

    @staticmethod
    def backward(ctx, dc):
        a, b = ctx.saved_tensors
        dc = _last_contiguous(dc)
        da = db = None
        if ctx.needs_input_grad[0]:
            da = _bmm(dc, b, trans_b=True, mantissa_bits=ctx.bits)     # dA = dC .^ B^T
        if ctx.needs_input_grad[1]:
            db = _bmm(a, dc, trans_a=True, mantissa_bits=ctx.bits)     # dB = A^T .^ dC
        return da, db, None


def pam_matmul(a: torch.Tensor, b: torch.Tensor, mantissa_bits: int = 23) -> torch.Tensor:
    """``a .^ b`` for 2-D or batched 3-D operands (leading batch dimension)."""
    _float32(a=a, b=b)
    if a.dim() == 2 and b.dim() == 2:
        return _PAMBmmFn.apply(a.unsqueeze(0), b.unsqueeze(0), int(mantissa_bits)).squeeze(0)
    if a.dim() == 3 and b.dim() == 3:
        return _PAMBmmFn.apply(a, b, int(mantissa_bits))
    raise ValueError("pam_matmul takes two 2-D or two 3-D tensors")


class PAMLinear(torch.nn.Module):
    """A linear layer whose products are PAM (forward and approximate-derivative backward)."""

    def __init__(self, in_features: int, out_features: int, bias: bool = True, device=None,
                 mantissa_bits: int = 23, derivative: str = "approximate"):
        super().__init__()
        self.in_features = in_features
        self.out_features = out_features
        self.mantissa_bits = mantissa_bits
        self.derivative = derivative
        self.weight = torch.nn.Parameter(torch.empty(out_features, in_features, device=device))
        self.bias = torch.nn.Parameter(torch.empty(out_features, device=device)) if bias else None
        self.reset_parameters()

    def reset_parameters(self) -> None:
        bound = 1.0 / math.sqrt(self.in_features) if self.in_features > 0 else 0.0
        with torch.no_grad():
            self.weight.uniform_(-bound, bound)
            if self.bias is not None:
                self.bias.uniform_(-bound, bound)

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        return pam_linear(x, self.weight, self.bias, self.mantissa_bits, self.derivative)

    def extra_repr(self) -> str:
        return (f"in_features={self.in_features}, out_features={self.out_features}, bias={self.bias is not None}, "
                f"mantissa_bits={self.mantissa_bits}, derivative={self.derivative}")
