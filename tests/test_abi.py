"""The C-ABI library on the host: it loads, exports every declared symbol and
rejects bad arguments before touching the GPU.  No compute calls."""
import ctypes
import os
import re

import pytest

import paper_2305_17190_amd as pam

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "pam.h")


def declared_functions():
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pam_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(pam.library_path()):
        pytest.skip("libpam.so not built (run __graft_entry__.build())")
    return pam.load()


def test_header_declares_the_boundary():
    names = declared_functions()
    for want in ("pam_mul", "pam_pad", "pam_palog2", "pam_paexp2", "pam_gemm", "pam_gemm_batched",
                 "pam_status_string", "pam_last_error"):
        assert want in names


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} declared in pam.h but not exported"
    assert set(pam.EXPORTS) == set(declared_functions())


def test_status_strings(lib):
    assert lib.pam_status_string(0) == b"PAM_SUCCESS"
    assert lib.pam_status_string(1) == b"PAM_ERROR_INVALID_VALUE"
    assert lib.pam_status_string(3) == b"PAM_ERROR_NOT_SUPPORTED"
    assert lib.pam_status_string(4) == b"PAM_ERROR_UNKNOWN"     # the library allocates nothing: no such status


def gemm_call(lib, **kw):
    a = dict(ta=0, tb=0, m=4, n=4, k=4, A=8, lda=4, B=8, ldb=4, C=8, ldc=4)
    a.update(kw)
    return lib.pam_gemm(a["ta"], a["tb"], a["m"], a["n"], a["k"], a["A"], a["lda"], a["B"], a["ldb"],
                        a["C"], a["ldc"], None)


@pytest.mark.parametrize("kw", [
    dict(m=-1), dict(n=-2), dict(k=-3), dict(ta=2), dict(tb=7),
    dict(lda=3), dict(ldb=3), dict(ldc=3), dict(ta=1, lda=3, m=4),
    dict(A=None), dict(B=None), dict(C=None), dict(m=1 << 31),
])
def test_gemm_rejects_bad_arguments(lib, kw):
    assert gemm_call(lib, **kw) == 1
    assert lib.pam_last_error() != b""


def test_batched_rejects_negative_stride_and_batch(lib):
    i = lib.pam_gemm_batched(0, 0, 4, 4, 4, 8, 4, -1, 8, 4, 16, 8, 4, 16, 2, None)
    assert i == 1
    assert lib.pam_gemm_batched(0, 0, 4, 4, 4, 8, 4, 16, 8, 4, 16, 8, 4, 16, -1, None) == 1


def test_empty_products_launch_nothing(lib):
    # m == 0 / n == 0 / batch == 0 succeed without any device work or pointers.
    assert gemm_call(lib, m=0, A=None, C=None, lda=4) == 0
    assert gemm_call(lib, n=0, B=None, C=None, ldb=1, ldc=1) == 0
    assert lib.pam_gemm_batched(0, 0, 4, 4, 4, None, 4, 0, None, 4, 0, None, 4, 0, 0, None) == 0
    assert lib.pam_mul(None, None, None, 0, None) == 0
    assert lib.pam_mul(None, None, None, -1, None) == 1
    assert lib.pam_pad(None, None, None, 0, None) == 0
    assert lib.pam_pad(None, None, None, -1, None) == 1
    assert lib.pam_palog2(None, None, 0, None) == 0
    assert lib.pam_paexp2(None, None, -2, None) == 1


def test_narrow_entry_points_reject_bad_mantissa_bits(lib):
    for bits in (-1, 24, 99):
        assert lib.pam_gemm_narrow(0, 0, 4, 4, 4, 8, 4, 0, 8, 4, 0, 8, 4, 0, 1, bits, None) == 1
        assert lib.pam_round_mantissa(8, 8, 4, bits, None) == 1
    assert lib.pam_round_mantissa(None, None, 0, 7, None) == 0
    assert lib.pam_gemm_narrow(0, 0, 0, 4, 4, None, 4, 0, 8, 4, 0, None, 4, 0, 1, 7, None) == 0
    assert lib.pam_gemm_narrow(0, 0, 4, 4, 4, 8, 3, 0, 8, 4, 0, 8, 4, 0, 1, 7, None) == 1   # lda < k


def test_elementwise_rejects_null_pointers(lib):
    assert lib.pam_mul(None, 8, 8, 4, None) == 1
    assert lib.pam_pad(8, None, 8, 4, None) == 1
    assert lib.pam_palog2(8, None, 4, None) == 1
    assert lib.pam_paexp2(None, 8, 4, None) == 1
    assert lib.pam_last_error() != b""


def test_plan_selection_is_host_logic(lib):
    # Large products use the 128x128 tile (three workgroups per compute
    # unit, 768 slots); 4096 tiles are five full rounds and 256 more: those
    # last tiles are K-split so they fill the last round, the rest keep K
    # whole.
    tm, tn, s, kg, whole = pam.plan(16384, 4096, 4096)
    assert (tm, tn, kg) == (128, 128, 1) and s > 1 and whole == 5 * 768
    # 1024 tiles on 768 slots would leave a last round on a third of the
    # slots: K is split (for every tile, or for the last round's tiles while
    # the first round takes the whole K) so the workgroups fill whole rounds.
    tm, tn, s, kg, whole = pam.plan(4096, 4096, 16384)
    assert (tm, tn, kg) == (128, 128, 1) and 2 <= s <= 16 and whole in (0, 768)
    assert pam.plan(8192, 2048, 512)[:2] == (128, 128)
    # Narrow outputs with long K split K; short-K batched narrow outputs get
    # more workgroups than 128x128 tiles would give (smaller tiles, K slices
    # or k-groups).
    assert pam.plan(8192, 512, 2048)[2] > 1
    assert pam.plan(768, 192, 12608)[2] >= 16
    tm, tn, s, kg, whole = pam.plan(256, 64, 256, 256)
    assert (tm, tn) != (128, 128) and (s > 1 or kg > 1)
    for m, n, k, b in ((1, 1, 1, 1), (5, 7, 3, 1), (300, 1, 17, 1), (16, 16, 100000, 1), (64, 64, 0, 3)):
        tm, tn, s, kg, whole = pam.plan(m, n, k, b)
        assert (tm, tn, kg) in ((128, 128, 1), (128, 64, 1), (128, 64, 2), (64, 64, 1), (64, 64, 4))
        assert 1 <= s <= 64 and whole >= 0
    with pytest.raises(pam.PamError):
        pam.plan(0, 4, 4)


@pytest.mark.parametrize("plan", [(96, 64, 1, 1), (128, 128, 0, 1), (128, 128, 1, 4), (64, 64, 1, 2),
                                  (64, 64, 65, 1), (128, 128, 2, 1, -1)])
def test_with_plan_rejects_bad_tiles(lib, plan):
    P = pam._Plan(*plan)
    assert lib.pam_gemm_batched_with_plan(0, 0, 4, 4, 4, 8, 4, 16, 8, 4, 16, 8, 4, 16, 1, ctypes.byref(P),
                                          None, 0, None) == 1
    out = ctypes.c_size_t()
    assert lib.pam_gemm_plan_workspace_size(4, 4, 4, 1, ctypes.byref(P), ctypes.byref(out)) == 1


def test_with_plan_split_needs_its_workspace(lib):
    """A forced split plan takes its partial sums from the caller: its size is
    splits x split tiles x tile, and a smaller or missing workspace is refused
    before any launch (fake, never dereferenced pointers)."""
    m, n, k = 300, 200, 4000
    out = ctypes.c_size_t()
    P = pam._Plan(128, 64, 4, 1, 0)
    assert lib.pam_gemm_plan_workspace_size(m, n, k, 1, ctypes.byref(P), ctypes.byref(out)) == 0
    assert out.value == 4 * 3 * 4 * 128 * 64 * 4
    args = (0, 0, m, n, k, 256, k, 0, 256, n, 0, 256, n, 0, 1, ctypes.byref(P))
    assert lib.pam_gemm_batched_with_plan(*args, None, 0, None) == 1
    assert b"smaller" in lib.pam_last_error()
    assert lib.pam_gemm_batched_with_plan(*args, 4096, out.value - 1, None) == 1
    assert lib.pam_gemm_batched_with_plan(*args, 4100, out.value, None) == 1
    assert b"aligned" in lib.pam_last_error()
    P1 = pam._Plan(128, 64, 1, 1, 0)
    assert lib.pam_gemm_plan_workspace_size(m, n, k, 1, ctypes.byref(P1), ctypes.byref(out)) == 0
    assert out.value == 0
    # hybrid: the first 10 of 12 tiles whole, the last 2 in 4 slices
    P2 = pam._Plan(128, 64, 4, 1, 10)
    assert lib.pam_gemm_plan_workspace_size(m, n, k, 1, ctypes.byref(P2), ctypes.byref(out)) == 0
    assert out.value == 4 * 2 * 128 * 64 * 4


def test_leading_dimension_limit(lib):
    for big in (1 << 23, 1 << 22):
        for kw in (dict(lda=big), dict(ldb=big)):
            assert gemm_call(lib, **kw) == 3
            assert b"2^22" in lib.pam_last_error()
    # Just below the limit the arguments are valid (the call then fails only
    # for want of a device here, with another message).
    gemm_call(lib, lda=(1 << 22) - 4, ldb=(1 << 22) - 4)
    assert b"2^22" not in lib.pam_last_error()


def test_binding_refuses_cpu_tensors():
    torch = pytest.importorskip("torch")
    a = torch.ones(8)
    with pytest.raises(pam.PamError):
        pam.mul(a, a)
    with pytest.raises(pam.PamError):
        pam.gemm(torch.ones(2, 2), torch.ones(2, 2))
    for fn in (pam.palog2, pam.paexp2):
        with pytest.raises(pam.PamError):
            fn(a)
    with pytest.raises(pam.PamError):
        pam.pad(a, a)


def test_autograd_wrappers_refuse_cpu_tensors():
    torch = pytest.importorskip("torch")
    from paper_2305_17190_amd.autograd import PAMLinear, pam_matmul
    lin = PAMLinear(4, 3)
    with pytest.raises(pam.PamError):
        lin(torch.ones(2, 4))
    with pytest.raises(pam.PamError):
        pam_matmul(torch.ones(2, 2), torch.ones(2, 2))
    # float32 only (the gradients are float32 products), refused before any call
    with pytest.raises(TypeError):
        lin(torch.ones(2, 4, dtype=torch.bfloat16))
    with pytest.raises(TypeError):
        pam_matmul(torch.ones(2, 2, dtype=torch.float64), torch.ones(2, 2))


def test_exact_grad_rejects_bad_arguments(lib):
    # transA N: lda >= k, ldb >= n, ldm >= n, ldc >= n
    assert lib.pam_gemm_exact_grad(0, 4, 4, 4, 8, 4, 8, 4, 8, 3, 8, 4, None) == 1      # ldm < n
    assert lib.pam_gemm_exact_grad(0, 4, 4, 4, 8, 3, 8, 4, 8, 4, 8, 4, None) == 1      # lda < k
    assert lib.pam_gemm_exact_grad(0, 4, 4, 4, 8, 4, 8, 4, None, 4, 8, 4, None) == 1   # Mod NULL
    assert lib.pam_gemm_exact_grad(2, 4, 4, 4, 8, 4, 8, 4, 8, 4, 8, 4, None) == 1      # bad transA
    assert lib.pam_gemm_exact_grad(0, 0, 4, 4, None, 4, 8, 4, None, 4, None, 4, None) == 0   # m == 0


def _ws_size(lib, m, n, k, batch=1):
    out = ctypes.c_size_t(12345)
    st = lib.pam_gemm_workspace_size(m, n, k, batch, ctypes.byref(out))
    return st, out.value


def test_workspace_size_follows_the_plan(lib):
    # Zero when the plan keeps K whole, splits x split tiles x tile otherwise.
    for m, n, k, b in ((16384, 4096, 4096, 1), (4096, 4096, 16384, 1), (768, 192, 12608, 1), (256, 64, 256, 256),
                       (5, 7, 3, 1), (8192, 2048, 512, 1)):
        tm, tn, s, kg, whole = pam.plan(m, n, k, b)
        st, got = _ws_size(lib, m, n, k, b)
        assert st == 0
        tiles = -(-m // tm) * -(-n // tn) * b
        split_tiles = 0 if s == 1 else (tiles - whole if whole else tiles)
        assert got == s * split_tiles * tm * tn * 4, (m, n, k, b)
    assert _ws_size(lib, 0, 5, 5) == (0, 0)
    assert _ws_size(lib, 5, 5, 0) == (0, 0)
    assert _ws_size(lib, -1, 5, 5)[0] == 1
    assert lib.pam_gemm_workspace_size(4, 4, 4, 1, None) == 1
    out = ctypes.c_size_t(7)
    assert lib.pam_gemm_exact_grad_workspace_size(4096, 4096, 16384, ctypes.byref(out)) == 0 and out.value == 0
    assert lib.pam_gemm_exact_grad_workspace_size(256, 256, 16384, ctypes.byref(out)) == 0
    assert out.value > 0 and out.value % (256 * 256 * 4) == 0
    assert lib.pam_gemm_exact_grad_workspace_size(4, 4, 4, None) == 1


def _gemm_ws(lib, m, n, k, ws, ws_bytes, bits=23):
    # Fake, never dereferenced device pointers: every case fails validation
    # before any launch.
    return lib.pam_gemm_batched_ws(0, 0, m, n, k, 256, k, 0, 256, n, 0, 256, n, 0, 1, bits, ws, ws_bytes, None)


def test_workspace_entry_point_rejects_bad_workspaces(lib):
    m, n, k = 768, 192, 12608                    # a split-K plan
    st, need = _ws_size(lib, m, n, k)
    assert st == 0 and need > 0
    assert _gemm_ws(lib, m, n, k, 4096, need - 4) == 1
    assert b"smaller" in lib.pam_last_error()
    assert _gemm_ws(lib, m, n, k, None, need) == 1
    assert b"NULL" in lib.pam_last_error()
    assert _gemm_ws(lib, m, n, k, 4096 + 4, need) == 1
    assert b"aligned" in lib.pam_last_error()
    assert _gemm_ws(lib, m, n, k, 4096, need, bits=24) == 1
    # exact-derivative product: a long-K, few-tile shape needs a workspace
    out = ctypes.c_size_t()
    assert lib.pam_gemm_exact_grad_workspace_size(256, 256, 16384, ctypes.byref(out)) == 0
    assert lib.pam_gemm_exact_grad_ws(0, 256, 256, 16384, 256, 16384, 256, 256, 256, 256, 256, 256,
                                      4096, out.value - 4, None) == 1
    assert b"smaller" in lib.pam_last_error()


def test_absurd_batch_is_refused_not_overflowed(lib):
    # tiles x batch beyond 2^62: refused with a message, before any device call
    st, _ = _ws_size(lib, 1 << 30, 1 << 30, 64, 1 << 40)
    assert st == 1 and b"too many" in lib.pam_last_error()
    assert lib.pam_gemm_batched(0, 0, 4, 4, 4, 8, 4, 16, 8, 4, 16, 8, 4, 16, 1 << 62, None) == 1
    # every planning entry point applies the same bound (2^40 output tiles of 64 x 64)
    with pytest.raises(pam.PamError, match="too many"):
        pam.plan(1 << 30, 1 << 30, 64, 1 << 40)
    with pytest.raises(pam.PamError, match="below 2"):
        pam.plan(1 << 31, 4, 4)
    # a large but launchable product (2^20 tiles of 128 x 128 per matrix) is planned
    assert pam.plan(1 << 17, 1 << 17, 64, 4)[:2] in {(128, 128), (128, 64), (64, 64)}
    assert _ws_size(lib, 1 << 17, 1 << 17, 64, 4)[0] == 0
