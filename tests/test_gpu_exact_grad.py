"""Exact-derivative products (Table 1, reading R15) on the GPU against the
oracle, directly and through pam_linear(derivative="exact")."""
import numpy as np
import pytest

import pam_workloads as wl
import paper_2305_17190_amd as pam
from gpu_util import check_gemm, device, note, to_dev
from oracle import pam_ref

pytestmark = pytest.mark.gpu


def operands(t, n, k, seed, edges=False):
    g = np.random.default_rng(seed)
    x = g.standard_normal((t, k)).astype(np.float32)
    w = (g.standard_normal((n, k)) * 0.05).astype(np.float32)
    dy = (g.standard_normal((t, n)) * 1e-3).astype(np.float32)
    if edges:
        for arr, s in ((x, 1), (w, 2), (dy, 3)):
            flat = arr.reshape(-1)
            idx = g.choice(flat.size, size=max(4, flat.size // 100), replace=False)
            kinds = g.integers(0, 4, size=idx.size)
            flat[idx] = np.where(kinds == 0, 0.0, np.where(kinds == 1, -0.0, np.where(
                kinds == 2, 1e-40 * s, 1.5 * 2.0 ** -120))).astype(np.float32)
    return x, w, dy


@pytest.mark.parametrize("t,n,k,edges", [(150, 70, 97, False), (150, 70, 97, True), (64, 128, 128, False),
                                         (3000, 40, 33, True), (1, 1, 1, False), (300, 5, 260, True)])
def test_exact_grads_match_oracle(t, n, k, edges):
    note(f"exact grads T={t} N={n} K={k} edges={edges}")
    x, w, dy = operands(t, n, k, 800 + t + n + k, edges)
    dxo, sdx, dwo, sdw = pam_ref.pam_exact_grads_ref(dy, x, w)
    xd, wd, dyd = to_dev(x), to_dev(w), to_dev(dy)
    dx = pam.exact_grad(dyd, wd, xd).cpu().numpy()
    dw = pam.exact_grad(dyd, xd, wd, trans_a=True).cpu().numpy()
    check_gemm(dx, dxo, sdx, n, "dX")
    check_gemm(dw, dwo, sdw, t, "dW")


def test_power_of_two_weights_give_the_plain_matmul():
    """With W = +-2^e every term is exact and dX = dY W exactly in float64;
    the GPU sum must be within float32 rounding of it."""
    note("exact dX with power-of-two weights")
    g = np.random.default_rng(810)
    x = g.standard_normal((90, 50)).astype(np.float32)
    w = (np.where(g.random((40, 50)) < 0.5, -1.0, 1.0) * np.ldexp(1.0, g.integers(-6, 6, (40, 50)))).astype(np.float32)
    dy = g.standard_normal((90, 40)).astype(np.float32)
    dx = pam.exact_grad(to_dev(dy), to_dev(w), to_dev(x)).cpu().numpy()
    ref = dy.astype(np.float64) @ w.astype(np.float64)
    s = np.abs(dy.astype(np.float64)) @ np.abs(w.astype(np.float64))
    check_gemm(dx, ref, s, 40, "dX = dY W")


def test_pam_linear_exact_derivative():
    import torch
    from paper_2305_17190_amd.autograd import pam_linear
    note("pam_linear derivative=exact forward + backward")
    dev = device()
    x, w, dy = operands(130, 60, 80, 811)
    xt = torch.from_numpy(x).to(dev).requires_grad_()
    wt = torch.from_numpy(w).to(dev).requires_grad_()
    y = pam_linear(xt, wt, derivative="exact")
    y.backward(torch.from_numpy(dy).to(dev))
    c, s = pam_ref.pam_gemm_ref(x, w, False, True)
    check_gemm(y.detach().cpu().numpy(), c, s, 80, "Y")
    dxo, sdx, dwo, sdw = pam_ref.pam_exact_grads_ref(dy, x, w)
    check_gemm(xt.grad.cpu().numpy(), dxo, sdx, 60, "dX exact")
    check_gemm(wt.grad.cpu().numpy(), dwo, sdw, 130, "dW exact")


def test_workload5_exact_dx_sampled_rows():
    """w5's dX with the exact derivative (16384 x 4096 x 4096), 4 sampled rows."""
    note("w5 exact dX, 4 sampled rows")
    host = wl.workload_inputs(5, only=["X", "W", "dY"])
    x, w, dy = host["X"], host["W"], host["dY"]
    dx = pam.exact_grad(to_dev(dy), to_dev(w), to_dev(x))
    rows = np.random.default_rng(812).choice(x.shape[0], size=4, replace=False)
    dxo, sdx, _, _ = pam_ref.pam_exact_grads_ref(dy[rows], x[rows], w)
    check_gemm(dx.cpu().numpy()[rows], dxo, sdx, 4096, "w5 exact dX")
