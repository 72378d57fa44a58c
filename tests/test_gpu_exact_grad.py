"""Exact-derivative products (Table 1, reading R15) on the GPU against the
oracle, directly and through pam_linear(derivative="exact"): ordinary
operands, every exponent region of every operand (zero / denormal, the safe
band, tiny and huge normals, products that underflow or saturate, the 2^128
factor), single-term and 16-term sums compared bit for bit, workgroups with
few and with many outputs whose X or W is tiny or huge, split K."""
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


def region_values(shape, g, lo_share=0.3, hi_share=0.3, zero_share=0.1):
    """float32 values whose exponent fields cover every region: the band
    [64, 190] where products cannot leave the normal range, tiny normals
    (1..63), huge normals (191..254), zeros and denormals."""
    u = g.random(shape)
    field = np.where(u < lo_share, g.integers(1, 64, shape),
                     np.where(u < lo_share + hi_share, g.integers(191, 255, shape), g.integers(64, 191, shape)))
    mant = g.integers(0, 1 << 23, shape)
    sign = g.integers(0, 2, shape)
    bits = (sign << 31) | (field << 23) | mant
    z = g.random(shape) < zero_share
    bits = np.where(z, np.where(g.random(shape) < 0.5, sign << 31, (sign << 31) | g.integers(1, 1 << 23, shape)), bits)
    return bits.astype(np.uint32).view(np.float32)


def small_dy(shape, g):
    """dY at most 2^-9 in magnitude (no term reaches FLT_MAX: factors are at
    most 2^128), down to the tiny normals, with zeros and denormals."""
    field = g.integers(1, 118, shape)
    bits = (g.integers(0, 2, shape) << 31) | (field << 23) | g.integers(0, 1 << 23, shape)
    bits = np.where(g.random(shape) < 0.05, g.integers(0, 1 << 23, shape), bits)
    return bits.astype(np.uint32).view(np.float32)


def check_single_terms(got, ref, what):
    """One term per output: the kernel's fma rounds the exact term once, so a
    normal result equals the float32 rounding of the exact value bit for bit;
    results below 2^-126 are flushed."""
    got = np.asarray(got, np.float32)
    with np.errstate(over="ignore"):
        ref32 = ref.astype(np.float32)
    normal = np.abs(ref32) >= np.float32(2.0 ** -126)
    assert np.array_equal(got[normal].view(np.uint32), ref32[normal].view(np.uint32)), what
    assert np.all(np.abs(got[~normal]) <= np.float32(2.0 ** -126)), what


@pytest.mark.parametrize("terms", [1, 16])
def test_every_region_short_sums(terms):
    """dX with N = terms and dW with T = terms (each output a sum of that many
    exact terms) over operands in every exponent region."""
    note(f"exact grads, every region, {terms}-term sums")
    g = np.random.default_rng(830 + terms)
    t, n, k = 300, terms, 260
    x = region_values((t, k), g)
    w = region_values((n, k), g)
    dy = small_dy((t, n), g)
    dxo, sdx, _, _ = pam_ref.pam_exact_grads_ref(dy, x, w)
    dx = pam.exact_grad(to_dev(dy), to_dev(w), to_dev(x)).cpu().numpy()
    check_gemm(dx, dxo, sdx, n, "dX")
    if terms == 1:
        check_single_terms(dx, dxo, "dX single terms")
    # dW: T = terms rows
    t2, n2 = terms, 290
    x2 = region_values((t2, k), g)
    w2 = region_values((n2, k), g)
    dy2 = small_dy((t2, n2), g)
    _, _, dwo, sdw = pam_ref.pam_exact_grads_ref(dy2, x2, w2)
    dw = pam.exact_grad(to_dev(dy2), to_dev(x2), to_dev(w2), trans_a=True).cpu().numpy()
    check_gemm(dw, dwo, sdw, t2, "dW")
    if terms == 1:
        check_single_terms(dw, dwo, "dW single terms")


def test_factor_two_to_the_128():
    """W = 1.5 2^127 with X = 1.75 2^-10: the carry takes the factor to 2^128
    while X .^ W = 1.25 2^118 is not clamped; dY = 2^-20 gives 2^108 exactly.
    With X = 1.75 the product saturates and the derivative is 0."""
    note("exact grad factor 2^128")
    x = np.float32([[1.75 * 2.0 ** -10, 1.75, -1.75 * 2.0 ** -10]])
    w = np.float32([[1.5 * 2.0 ** 127, 1.5 * 2.0 ** 127, -1.5 * 2.0 ** 127]])
    dy = np.float32([[2.0 ** -20]])
    dx = pam.exact_grad(to_dev(dy), to_dev(w), to_dev(x)).cpu().numpy()
    assert dx.tolist() == [[2.0 ** 108, 0.0, -2.0 ** 108]]
    dxo, _, _, _ = pam_ref.pam_exact_grads_ref(dy, x, w)
    assert dxo.tolist() == dx.tolist()


@pytest.mark.parametrize("share", [0.0005, 0.01, 0.2, 1.0])
def test_extreme_mod_shares(share):
    """X with this share of tiny / huge normals (a few per workgroup up to
    every output: the per-output sums and the all-general workgroups), W and
    dY ordinary, plus some tiny and huge W; split K for dW."""
    note(f"exact grads, extreme X share {share}")
    g = np.random.default_rng(840 + int(share * 1e4))
    t, n, k = 700, 96, 200
    x = g.standard_normal((t, k)).astype(np.float32)
    pick = g.random((t, k)) < share
    ext = region_values((t, k), g, lo_share=0.5, hi_share=0.5, zero_share=0.0)
    x = np.where(pick, ext, x)
    w = (g.standard_normal((n, k)) * 0.05).astype(np.float32)
    wpick = g.random((n, k)) < 0.002
    w = np.where(wpick, region_values((n, k), g, 0.5, 0.5, 0.0), w)
    dy = small_dy((t, n), g)
    dxo, sdx, dwo, sdw = pam_ref.pam_exact_grads_ref(dy, x, w)
    xd, wd, dyd = to_dev(x), to_dev(w), to_dev(dy)
    dx = pam.exact_grad(dyd, wd, xd).cpu().numpy()
    dw = pam.exact_grad(dyd, xd, wd, trans_a=True).cpu().numpy()
    check_gemm(dx, dxo, sdx, n, "dX")
    check_gemm(dw, dwo, sdw, t, "dW")


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
