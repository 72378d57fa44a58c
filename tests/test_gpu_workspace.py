"""The caller-workspace entry points against the allocating ones, through
the C ABI: the same plan, so bitwise equal results (split-K, hybrid and
unsplit plans, narrow mantissas, the exact-derivative product)."""
import ctypes

import numpy as np
import pytest

import paper_2305_17190_amd as pam
from gpu_util import device, note, to_dev

pytestmark = pytest.mark.gpu

SHAPES = [(768, 192, 12608, 1), (8192, 2048, 512, 1), (256, 64, 256, 16), (300, 260, 200, 2), (5, 7, 3, 1)]


@pytest.mark.parametrize("m,n,k,batch", SHAPES)
@pytest.mark.parametrize("bits", [23, 7])
def test_gemm_ws_equals_allocating_entry_point(m, n, k, batch, bits):
    import torch
    lib = pam.load()
    note(f"pam_gemm_batched_ws vs pam_gemm_narrow m={m} n={n} k={k} batch={batch} bits={bits} "
         f"plan={pam.plan(m, n, k, batch)}")
    g = np.random.default_rng(91)
    a = to_dev(g.standard_normal((batch, m, k)).astype(np.float32))
    b = to_dev(g.standard_normal((batch, k, n)).astype(np.float32))
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
    assert torch.equal(c1.view(torch.int32), c2.view(torch.int32))
    # and the binding (its own workspace) gives the same bits
    c3 = pam.bmm(a, b, mantissa_bits=bits)
    assert torch.equal(c3.view(torch.int32), c1.view(torch.int32))


@pytest.mark.parametrize("m,n,k,ta", [(256, 256, 4096, False), (192, 130, 3000, True), (300, 200, 100, False)])
def test_exact_grad_ws_equals_allocating_entry_point(m, n, k, ta):
    import torch
    lib = pam.load()
    note(f"pam_gemm_exact_grad_ws vs pam_gemm_exact_grad m={m} n={n} k={k} ta={ta}")
    g = np.random.default_rng(92)
    a = to_dev(g.standard_normal((k, m) if ta else (m, k)).astype(np.float32))
    b = to_dev(g.standard_normal((k, n)).astype(np.float32))
    mod = to_dev(g.standard_normal((m, n)).astype(np.float32))
    c1 = torch.full((m, n), float("nan"), device=device())
    c2 = torch.full((m, n), float("nan"), device=device())
    size = ctypes.c_size_t()
    assert lib.pam_gemm_exact_grad_workspace_size(m, n, k, ctypes.byref(size)) == 0
    ws = torch.empty(max(size.value, 1), dtype=torch.uint8, device=device())
    stream = torch.cuda.current_stream().cuda_stream
    lda = m if ta else k
    args = (1 if ta else 0, m, n, k, a.data_ptr(), lda, b.data_ptr(), n, mod.data_ptr(), n)
    assert lib.pam_gemm_exact_grad(*args, c1.data_ptr(), n, stream) == 0
    assert lib.pam_gemm_exact_grad_ws(*args, c2.data_ptr(), n, ws.data_ptr(), size.value, stream) == 0
    torch.cuda.synchronize()
    assert torch.equal(c1.view(torch.int32), c2.view(torch.int32))
    c3 = pam.exact_grad(a, b, mod, trans_a=ta)
    assert torch.equal(c3.view(torch.int32), c1.view(torch.int32))
