"""The workspace contract of the C ABI: the library allocates nothing.

* Entry points with a caller workspace (pam_gemm_batched_ws, the binding's
  path) run the library's plan, split K included, bitwise equal to the same
  plan forced through pam_gemm_batched_with_plan.
* Entry points without one (pam_gemm, pam_gemm_batched, pam_gemm_narrow,
  pam_gemm_exact_grad) run the plan pam_gemm_plan_for_workspace(..., 0)
  names, which never splits K, bitwise equal to that plan forced.
* Their host calls return while the product's kernels still run: a long
  split-shape product's completion event is still pending right after the
  call, and the call took well under the product's GPU time.
"""
import ctypes
import time

import numpy as np
import pytest

import paper_2305_17190_amd as pam
from gpu_util import check_gemm, device, note, oracle_gemm, to_dev

pytestmark = pytest.mark.gpu

SHAPES = [(768, 192, 12608, 1), (8192, 2048, 512, 1), (256, 64, 256, 16), (300, 260, 200, 2), (5, 7, 3, 1),
          (4096, 1024, 4096, 1)]


def forced(a, b, m, n, k, batch, plan):
    """The product under an explicit plan (workspace from torch)."""
    c = pam.bmm(a, b, plan=plan)
    return c


@pytest.mark.parametrize("m,n,k,batch", SHAPES)
@pytest.mark.parametrize("bits", [23, 7])
def test_workspace_and_no_workspace_plans(m, n, k, batch, bits):
    import torch
    lib = pam.load()
    ws_plan = pam.plan(m, n, k, batch)
    free_plan = pam.plan(m, n, k, batch, max_workspace_bytes=0)
    note(f"workspace plans m={m} n={n} k={k} batch={batch} bits={bits} ws={ws_plan} none={free_plan}")
    assert free_plan[2] == 1
    g = np.random.default_rng(91)
    a = to_dev(g.standard_normal((batch, m, k)).astype(np.float32))
    b = to_dev(g.standard_normal((batch, k, n)).astype(np.float32))
    if bits != 23:
        a, b = pam.round_mantissa(a, bits), pam.round_mantissa(b, bits)
    c1 = torch.full((batch, m, n), float("nan"), device=device())
    c2 = torch.full((batch, m, n), float("nan"), device=device())
    size = ctypes.c_size_t()
    assert lib.pam_gemm_workspace_size(m, n, k, batch, ctypes.byref(size)) == 0
    ws = torch.empty(max(size.value, 1), dtype=torch.uint8, device=device())
    stream = torch.cuda.current_stream().cuda_stream
    common = (0, 0, m, n, k, a.data_ptr(), k, m * k, b.data_ptr(), n, k * n)
    assert lib.pam_gemm_narrow(*common, c1.data_ptr(), n, m * n, batch, bits, stream) == 0
    assert lib.pam_gemm_batched_ws(*common, c2.data_ptr(), n, m * n, batch, bits, ws.data_ptr(), size.value,
                                   stream) == 0
    torch.cuda.synchronize()
    # operands already on the grid: rounding them again changes nothing
    assert torch.equal(c1.view(torch.int32), forced(a, b, m, n, k, batch, free_plan).view(torch.int32))
    assert torch.equal(c2.view(torch.int32), forced(a, b, m, n, k, batch, ws_plan).view(torch.int32))
    # and the binding (its own workspace) gives the workspace plan's bits
    c3 = pam.bmm(a, b, mantissa_bits=bits)
    assert torch.equal(c3.view(torch.int32), c2.view(torch.int32))
    if m * n * k * batch <= 1 << 27:
        an, bn = a.cpu().numpy(), b.cpu().numpy()
        c_ref, s_ref = oracle_gemm(an, bn, False, False, m, n, k, k, n, m * k, k * n,
                                   batches=list(range(batch)))
        check_gemm(c1.cpu().numpy(), c_ref, s_ref, k, "no-workspace plan")


@pytest.mark.parametrize("m,n,k,ta", [(256, 256, 4096, False), (192, 130, 3000, True), (300, 200, 100, False)])
def test_exact_grad_with_and_without_workspace(m, n, k, ta):
    """Split (workspace) and unsplit (none) exact-derivative products: both
    within float32 summation order of each other, the binding's equal to
    the workspace entry point's bit for bit."""
    import torch
    from oracle import pam_ref
    lib = pam.load()
    note(f"pam_gemm_exact_grad_ws vs pam_gemm_exact_grad m={m} n={n} k={k} ta={ta}")
    g = np.random.default_rng(92)
    a = g.standard_normal((k, m) if ta else (m, k)).astype(np.float32)
    b = g.standard_normal((k, n)).astype(np.float32)
    mod = g.standard_normal((m, n)).astype(np.float32)
    ad, bd, modd = to_dev(a), to_dev(b), to_dev(mod)
    c1 = torch.full((m, n), float("nan"), device=device())
    c2 = torch.full((m, n), float("nan"), device=device())
    size = ctypes.c_size_t()
    assert lib.pam_gemm_exact_grad_workspace_size(m, n, k, ctypes.byref(size)) == 0
    ws = torch.empty(max(size.value, 1), dtype=torch.uint8, device=device())
    stream = torch.cuda.current_stream().cuda_stream
    lda = m if ta else k
    args = (1 if ta else 0, m, n, k, ad.data_ptr(), lda, bd.data_ptr(), n, modd.data_ptr(), n)
    assert lib.pam_gemm_exact_grad(*args, c1.data_ptr(), n, stream) == 0
    assert lib.pam_gemm_exact_grad_ws(*args, c2.data_ptr(), n, ws.data_ptr(), size.value, stream) == 0
    torch.cuda.synchronize()
    c3 = pam.exact_grad(ad, bd, modd, trans_a=ta)
    assert torch.equal(c3.view(torch.int32), c2.view(torch.int32))
    # the oracle: dX form with dY = op(A), W = B, X = Mod
    dy = a.T if ta else a
    dxo, sdx, _, _ = pam_ref.pam_exact_grads_ref(np.ascontiguousarray(dy), mod, b)
    check_gemm(c1.cpu().numpy(), dxo, sdx, k, "exact grad, no workspace")
    check_gemm(c2.cpu().numpy(), dxo, sdx, k, "exact grad, workspace")


def test_host_calls_do_not_wait_for_the_gpu():
    """A split-shape product (w5's dW shape, ~10 ms on the GPU) through every
    entry point: each call returns while its kernels run."""
    import torch
    lib = pam.load()
    m, n, k = 4096, 4096, 16384
    note(f"asynchronous host calls, m={m} n={n} k={k}")
    assert pam.plan(m, n, k)[2] > 1          # the workspace plan splits K
    g = torch.Generator(device="cpu").manual_seed(93)
    a = torch.randn((k, m), generator=g).to(device())
    b = torch.randn((k, n), generator=g).to(device())
    mod = torch.randn((m, n), generator=g).to(device())
    c = torch.empty((m, n), device=device())
    size = ctypes.c_size_t()
    assert lib.pam_gemm_workspace_size(m, n, k, 1, ctypes.byref(size)) == 0 and size.value > 0
    ws = torch.empty(size.value, dtype=torch.uint8, device=device())
    esize = ctypes.c_size_t()
    assert lib.pam_gemm_exact_grad_workspace_size(m, n, k, ctypes.byref(esize)) == 0
    ews = torch.empty(max(esize.value, 1), dtype=torch.uint8, device=device())
    stream = torch.cuda.current_stream().cuda_stream
    calls = {
        "pam_gemm": lambda: lib.pam_gemm(1, 0, m, n, k, a.data_ptr(), m, b.data_ptr(), n, c.data_ptr(), n, stream),
        "pam_gemm_batched": lambda: lib.pam_gemm_batched(1, 0, m, n, k, a.data_ptr(), m, 0, b.data_ptr(), n, 0,
                                                         c.data_ptr(), n, 0, 1, stream),
        "pam_gemm_narrow": lambda: lib.pam_gemm_narrow(1, 0, m, n, k, a.data_ptr(), m, 0, b.data_ptr(), n, 0,
                                                       c.data_ptr(), n, 0, 1, 7, stream),
        "pam_gemm_batched_ws": lambda: lib.pam_gemm_batched_ws(1, 0, m, n, k, a.data_ptr(), m, 0, b.data_ptr(), n,
                                                               0, c.data_ptr(), n, 0, 1, 23, ws.data_ptr(),
                                                               size.value, stream),
        "pam_gemm_exact_grad": lambda: lib.pam_gemm_exact_grad(1, m, n, k, a.data_ptr(), m, b.data_ptr(), n,
                                                               mod.data_ptr(), n, c.data_ptr(), n, stream),
        "pam_gemm_exact_grad_ws": lambda: lib.pam_gemm_exact_grad_ws(1, m, n, k, a.data_ptr(), m, b.data_ptr(), n,
                                                                     mod.data_ptr(), n, c.data_ptr(), n,
                                                                     ews.data_ptr(), esize.value, stream),
    }
    for name, call in calls.items():
        call()                                  # first call: device check, code object load
        torch.cuda.synchronize()
        done = torch.cuda.Event()
        t0 = time.perf_counter()
        assert call() == 0, name
        host_s = time.perf_counter() - t0
        done.record()
        pending = not done.query()
        torch.cuda.synchronize()
        note(f"{name}: host call {host_s * 1e3:.3f} ms, kernels pending after it: {pending}")
        assert pending, f"{name}: the product had finished when its call returned"
        assert host_s < 2e-3, f"{name}: the host call took {host_s * 1e3:.2f} ms"
