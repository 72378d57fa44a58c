"""pam_gemm_batched_noalloc, the entry point for callers that cannot allocate:
through the C ABI against pam_gemm_batched_ws (the same product with a
caller workspace) on calls in a row, each later one smaller, so every call
after the first finds the scratch holding the previous call's partial sums.
Where the library's plan fits the 64 MiB scratch the two entry points run the
same plan and must agree bit for bit; where it does not (w5's weight-gradient
shape), the no-alloc call runs the fastest plan that fits, which must equal
that plan forced with a caller workspace bit for bit and the oracle within
the tolerance."""
import ctypes

import numpy as np
import pytest

import paper_2305_17190_amd as pam
from gpu_util import check_gemm, device, note, oracle_gemm, to_dev

pytestmark = pytest.mark.gpu

SCRATCH = 64 << 20


def ws_product(lib, a, b, m, n, k, batch, stream, bits=23):
    import torch
    size = ctypes.c_size_t()
    assert lib.pam_gemm_workspace_size(m, n, k, batch, ctypes.byref(size)) == 0
    ws = torch.empty(max(size.value, 1), dtype=torch.uint8, device=device())
    c = torch.full((batch, m, n), float("nan"), device=device())
    assert lib.pam_gemm_batched_ws(0, 0, m, n, k, a.data_ptr(), k, m * k, b.data_ptr(), n, k * n, c.data_ptr(), n,
                                   m * n, batch, bits, ws.data_ptr(), size.value, stream) == 0
    return c, size.value


def noalloc_product(lib, a, b, m, n, k, batch, stream, bits=23):
    import torch
    c = torch.full((batch, m, n), float("nan"), device=device())
    st = lib.pam_gemm_batched_noalloc(0, 0, m, n, k, a.data_ptr(), k, m * k, b.data_ptr(), n, k * n, c.data_ptr(),
                                      n, m * n, batch, bits, stream)
    assert st == 0, lib.pam_last_error()
    return c


def operands(batch, m, n, k, seed):
    g = np.random.default_rng(seed)
    a = g.standard_normal((batch, m, k)).astype(np.float32)
    b = g.standard_normal((batch, k, n)).astype(np.float32)
    return a, b


def test_noalloc_matches_the_workspace_entry_point():
    import torch
    lib = pam.load()
    stream = torch.cuda.current_stream().cuda_stream
    # three calls, each smaller than the one before, all with split plans that fit the scratch
    for (m, n, k, batch, bits, seed) in ((768, 192, 12608, 1, 23, 1), (300, 260, 5000, 2, 23, 2),
                                         (130, 70, 3000, 1, 7, 3)):
        plan = pam.plan(m, n, k, batch)
        note(f"noalloc vs ws m={m} n={n} k={k} batch={batch} bits={bits} plan={plan}")
        a, b = operands(batch, m, n, k, seed)
        ad, bd = to_dev(a), to_dev(b)
        c_ws, need = ws_product(lib, ad, bd, m, n, k, batch, stream, bits)
        assert plan[2] > 1 and 0 < need <= SCRATCH
        assert pam.plan(m, n, k, batch, max_workspace_bytes=SCRATCH) == plan
        c_na = noalloc_product(lib, ad, bd, m, n, k, batch, stream, bits)
        torch.cuda.synchronize()
        assert torch.equal(c_na.view(torch.int32), c_ws.view(torch.int32)), (m, n, k, batch)
        if bits == 23:
            rows = np.unique(np.linspace(0, m - 1, 12).astype(np.int64))
            c_ref, s_ref = oracle_gemm(a, b, False, False, m, n, k, k, n, m * k, k * n,
                                       batches=list(range(batch)), rows=rows)
            check_gemm(c_na.cpu().numpy()[:, rows], c_ref, s_ref, k, "noalloc")


def test_noalloc_plan_within_the_scratch():
    """w5's dW shape: the library's plan needs 128 MiB of partial sums, so the
    no-alloc call runs the fastest plan whose partial sums fit in 64 MiB;
    then a smaller product reuses the scratch."""
    import torch
    lib = pam.load()
    stream = torch.cuda.current_stream().cuda_stream
    m, n, k = 4096, 4096, 16384
    full = pam.plan(m, n, k)
    fit = pam.plan(m, n, k, max_workspace_bytes=SCRATCH)
    note(f"noalloc within the scratch m={m} n={n} k={k}: library plan {full}, scratch plan {fit}")
    size = ctypes.c_size_t()
    assert lib.pam_gemm_workspace_size(m, n, k, 1, ctypes.byref(size)) == 0 and size.value > SCRATCH
    p = pam._Plan(*fit)
    need = ctypes.c_size_t()
    assert lib.pam_gemm_plan_workspace_size(m, n, k, 1, ctypes.byref(p), ctypes.byref(need)) == 0
    assert need.value <= SCRATCH
    g = torch.Generator(device="cpu").manual_seed(5)
    a = torch.randn((1, m, k), generator=g).to(device())
    b = torch.randn((1, k, n), generator=g).to(device())
    c_na = noalloc_product(lib, a, b, m, n, k, 1, stream)
    c_forced = pam.bmm(a, b, plan=fit)
    torch.cuda.synchronize()
    assert torch.equal(c_na.view(torch.int32), c_forced.view(torch.int32))
    rows = np.array([0, 1000, 3071, 4095])
    an, bn = a.cpu().numpy(), b.cpu().numpy()
    c_ref, s_ref = oracle_gemm(an, bn, False, False, m, n, k, k, n, rows=rows)
    check_gemm(c_na.cpu().numpy()[0][rows], c_ref[0], s_ref[0], k, "noalloc w5 dW rows")
    # a smaller split product right after, on the same scratch
    m2, n2, k2 = 200, 150, 9000
    a2, b2 = operands(1, m2, n2, k2, 6)
    ad2, bd2 = to_dev(a2), to_dev(b2)
    c_ws, need2 = ws_product(lib, ad2, bd2, m2, n2, k2, 1, stream)
    c_na2 = noalloc_product(lib, ad2, bd2, m2, n2, k2, 1, stream)
    torch.cuda.synchronize()
    assert need2 > 0
    assert torch.equal(c_na2.view(torch.int32), c_ws.view(torch.int32))


def test_noalloc_refuses_bad_arguments():
    lib = pam.load()
    assert lib.pam_gemm_batched_noalloc(0, 0, 4, 4, 4, 256, 3, 0, 256, 4, 0, 256, 4, 0, 1, 23, None) == 1
    assert lib.pam_gemm_batched_noalloc(0, 0, 4, 4, 4, 256, 4, 0, 256, 4, 0, 256, 4, 0, 1, 24, None) == 1
    assert lib.pam_gemm_batched_noalloc(0, 0, 0, 4, 4, None, 4, 0, 256, 4, 0, None, 4, 0, 1, 23, None) == 0
