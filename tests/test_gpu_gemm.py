"""PAM matrix products on the GPU against the CPU oracle, element by element.

Sizes span several tiles with ragged tails in every dimension.  The data
kinds drive each LDS encoding of the kernel: normal values (FAST), zeros,
denormals and underflowing products (GENERIC), and inf / NaN / |x| >= 2^64
(SPECIAL).  Every tiling and split-K setting is exercised through the
explicit-plan entry point.
"""
import numpy as np
import pytest

import paper_2305_17190_amd as pam
from gpu_util import check_gemm, device, note, oracle_gemm, to_dev
from oracle import pam_ref

pytestmark = pytest.mark.gpu

PLANS = [(128, 128, 1), (128, 64, 1), (128, 64, 1, 2), (64, 64, 1), (64, 64, 1, 4), (128, 128, 3), (128, 64, 7),
         (128, 64, 3, 2), (64, 64, 2), (64, 64, 3, 4),
         # whole-K tiles beside split ones in one launch
         (128, 128, 3, 1, 2), (128, 64, 7, 1, 1), (128, 64, 2, 2, 3), (64, 64, 2, 1, 5), (64, 64, 3, 4, 7),
         (64, 64, 5, 1, 11)]
TRANS = [(False, False), (False, True), (True, False), (True, True)]


def make(kind: str, shape, seed: int) -> np.ndarray:
    g = np.random.default_rng(seed)
    x = g.standard_normal(shape).astype(np.float32)
    flat = x.reshape(-1)
    n = flat.size
    if kind == "normal":
        return x
    if kind == "zeros_tiny":
        idx = g.choice(n, size=max(1, n // 25), replace=False)
        third = len(idx) // 3
        flat[idx[:third]] = np.where(g.random(third) < 0.5, 0.0, -0.0)
        flat[idx[third:2 * third]] = (g.uniform(0.5, 2.0, len(idx[third:2 * third])) * 2.0 ** -126).astype(np.float32)
        flat[idx[2 * third:]] = np.float32(3e-41)                       # denormal
        return x
    if kind == "underflow":
        e = g.integers(-75, -50, size=n)
        return (np.sign(flat) * np.ldexp(1.0 + np.abs(flat) % 1.0, e)).astype(np.float32).reshape(shape)
    if kind == "wide":
        e = g.integers(-70, 55, size=n)
        return (np.sign(flat) * np.ldexp(1.0 + np.abs(flat) % 1.0, e)).astype(np.float32).reshape(shape)
    if kind == "specials":
        idx = g.choice(n, size=max(3, n // 200), replace=False)
        vals = np.array([np.inf, -np.inf, np.nan, 2.0 ** 70, -(2.0 ** 65), 0.0], dtype=np.float32)
        flat[idx] = vals[g.integers(0, len(vals), size=len(idx))]
        return x
    raise ValueError(kind)


def run_case(m, n, k, ta, tb, kind_a, kind_b, plan=None, pad=(0, 0, 0), seed=0, batch=1):
    """Build op(A), op(B) with optional leading-dimension padding and compare."""
    a_rows, a_cols = (k, m) if ta else (m, k)
    b_rows, b_cols = (n, k) if tb else (k, n)
    a_buf = make(kind_a, (batch, a_rows, a_cols + pad[0]), seed)
    b_buf = make(kind_b, (batch, b_rows, b_cols + pad[1]), seed + 1)
    lda, ldb = a_cols + pad[0], b_cols + pad[1]
    ldc = n + pad[2]
    note(f"gemm m={m} n={n} k={k} ta={ta} tb={tb} A={kind_a} B={kind_b} plan={plan} pad={pad} batch={batch}")
    da = to_dev(a_buf)[:, :, :a_cols]
    db = to_dev(b_buf)[:, :, :b_cols]
    import torch
    c_full = torch.full((batch, m, ldc), float("nan"), device=device())
    c = c_full[:, :, :n]
    pam.bmm(da, db, trans_a=ta, trans_b=tb, out=c, plan=plan)
    got = c_full.cpu().numpy()
    if pad[2]:
        assert np.all(np.isnan(got[:, :, n:])), "wrote outside the output's columns"
    c_ref, s_ref = oracle_gemm(a_buf, b_buf, ta, tb, m, n, k, lda, ldb, a_buf[0].size, b_buf[0].size,
                               batches=list(range(batch)))
    check_gemm(got[:, :, :n], c_ref, s_ref, k, f"m={m} n={n} k={k} ta={ta} tb={tb} {kind_a}/{kind_b} {plan}")


@pytest.mark.parametrize("plan", PLANS, ids=lambda p: "x".join(map(str, p)))
@pytest.mark.parametrize("ta,tb", TRANS, ids=["NN", "NT", "TN", "TT"])
def test_plans_and_layouts_normal(plan, ta, tb):
    run_case(203, 150, 333, ta, tb, "normal", "normal", plan=plan, seed=11)


@pytest.mark.parametrize("ta,tb", TRANS, ids=["NN", "NT", "TN", "TT"])
@pytest.mark.parametrize("kinds", [("zeros_tiny", "normal"), ("normal", "zeros_tiny"), ("underflow", "underflow"),
                                   ("wide", "wide"), ("specials", "normal"), ("normal", "specials"),
                                   ("zeros_tiny", "specials")], ids=lambda k: "-".join(k))
def test_encodings(kinds, ta, tb):
    run_case(130, 200, 100, ta, tb, kinds[0], kinds[1], plan=(128, 64, 2), seed=21)
    run_case(130, 200, 100, ta, tb, kinds[0], kinds[1], plan=(64, 64, 1, 4), seed=22)


@pytest.mark.parametrize("pad", [(4, 4, 4), (1, 3, 5), (0, 0, 1)])
@pytest.mark.parametrize("ta,tb", TRANS, ids=["NN", "NT", "TN", "TT"])
def test_leading_dimension_padding(pad, ta, tb):
    run_case(77, 91, 64, ta, tb, "normal", "zeros_tiny", pad=pad, seed=31)


@pytest.mark.parametrize("mnk", [(1, 1, 1), (1, 300, 17), (300, 1, 17), (64, 64, 16), (129, 129, 1), (5, 7, 3),
                                 (256, 256, 4096), (16, 16, 2000)])
def test_shapes(mnk):
    m, n, k = mnk
    run_case(m, n, k, False, True, "normal", "normal", seed=41)


@pytest.mark.parametrize("ta,tb", TRANS, ids=["NN", "NT", "TN", "TT"])
def test_batched_strides(ta, tb):
    run_case(70, 40, 50, ta, tb, "normal", "zeros_tiny", batch=5, seed=51)


def test_batched_auto_plan_split():
    run_case(96, 64, 512, False, False, "normal", "normal", batch=3, seed=52)


@pytest.mark.parametrize("plan", [(64, 64, 3, 1, 3), (64, 64, 2, 4, 1), (128, 64, 4, 1, 4), (64, 64, 3, 1, 100),
                                  (64, 64, 3, 1, 9)], ids=lambda p: "x".join(map(str, p)))
def test_batched_whole_and_split_tiles(plan):
    # Two tiles per matrix, ten in all: the split tiles start inside a
    # matrix and run across the following ones; whole_tiles >= 10 splits none.
    run_case(70, 40, 150, False, True, "normal", "zeros_tiny", batch=5, seed=53, plan=plan)


def test_batched_broadcast_stride_zero():
    import torch
    note("bmm with a stride-0 (broadcast) B")
    g = np.random.default_rng(61)
    a = g.standard_normal((4, 33, 21)).astype(np.float32)
    b = g.standard_normal((21, 19)).astype(np.float32)
    db = to_dev(b).unsqueeze(0).expand(4, 21, 19)
    c = pam.bmm(to_dev(a), db).cpu().numpy()
    for z in range(4):
        c_ref, s_ref = pam_ref.pam_gemm_ref(a[z], b)
        check_gemm(c[z], c_ref, s_ref, 21, f"broadcast z={z}")


def test_identity_is_exact():
    note("gemm with B = I")
    g = np.random.default_rng(71)
    a = g.standard_normal((150, 140)).astype(np.float32)
    eye = np.eye(140, dtype=np.float32)
    for plan in PLANS:
        c = pam.bmm(to_dev(a[None]), to_dev(eye[None]), plan=plan).cpu().numpy()[0]
        assert np.array_equal(c.view(np.uint32), a.view(np.uint32)), f"identity not exact with plan {plan}"


def test_k1_equals_elementwise():
    note("gemm K = 1 equals broadcast pam_mul")
    g = np.random.default_rng(72)
    col = g.standard_normal((90, 1)).astype(np.float32)
    row = g.standard_normal((1, 70)).astype(np.float32)
    row[0, 3] = 0.0
    c = pam.gemm(to_dev(col), to_dev(row)).cpu().numpy()
    want = pam_ref.pam_mul_ref(np.repeat(col, 70, 1), np.repeat(row, 90, 0))
    assert np.array_equal(c, want)


@pytest.mark.parametrize("ta", [False, True], ids=["AN", "AT"])
@pytest.mark.parametrize("plan", [None, (128, 128, 1)], ids=["auto", "128x128"])
def test_leading_dimensions_near_the_limit(ta, plan):
    # lda = ldb = 2^22 - 4, the largest multiple of 4 the library takes: in a
    # 128-row panel the kernels' 32-bit per-thread byte offsets reach ~2.1 GB.
    # m = 130 crosses a panel; only the first columns of each row are used.
    ld = (1 << 22) - 4
    m, n, k = 130, 3, 5
    g = np.random.default_rng(81)
    a_rows, a_cols = (k, m) if ta else (m, k)
    a_buf = np.zeros((a_rows, ld), np.float32)
    a_buf[:, :a_cols] = g.standard_normal((a_rows, a_cols))
    b_buf = np.zeros((k, ld), np.float32)
    b_buf[:, :n] = g.standard_normal((k, n))
    note(f"gemm lda=ldb={ld} m={m} n={n} k={k} ta={ta} plan={plan}")
    da = to_dev(a_buf)[:, :a_cols]
    db = to_dev(b_buf)[:, :n]
    if plan is None:
        c = pam.gemm(da, db, trans_a=ta).cpu().numpy()
    else:
        c = pam.bmm(da.unsqueeze(0), db.unsqueeze(0), trans_a=ta, plan=plan).cpu().numpy()[0]
    del da, db
    c_ref, s_ref = oracle_gemm(a_buf, b_buf, ta, False, m, n, k, ld, ld)
    check_gemm(c, c_ref[0], s_ref[0], k, f"lda=ldb={ld} ta={ta} plan={plan}")


def test_long_k_many_slices():
    # K ~ 1e6 (odd) on a 3 x 5 output: the plan splits K into many slices.
    m, n, k = 3, 5, 1_000_003
    g = np.random.default_rng(82)
    a = g.standard_normal((m, k)).astype(np.float32)
    b = g.standard_normal((k, n)).astype(np.float32)
    tm, tn, splits, kg, whole = pam.plan(m, n, k)
    note(f"gemm m={m} n={n} k={k} plan={(tm, tn, splits, kg, whole)}")
    assert splits >= 16
    c = pam.gemm(to_dev(a), to_dev(b)).cpu().numpy()
    c_ref, s_ref = oracle_gemm(a, b, False, False, m, n, k, k, n)
    check_gemm(c, c_ref[0], s_ref[0], k, "long K")


def test_batch_beyond_one_launch():
    # 2^24 + 3 one-element products: more workgroups than one launch may hold
    # (2^24 - 1), so the library issues two launches; every product is a K = 1
    # sum, i.e. pam_mul of the two elements.
    import pam_workloads as wl
    n = (1 << 24) + 3
    note(f"bmm batch={n} of 1x1x1 products (two launches)")
    a, b = wl.pam_mul_inputs(n, 75)
    c = pam.bmm(to_dev(a.reshape(n, 1, 1)), to_dev(b.reshape(n, 1, 1))).cpu().numpy().reshape(n)
    want = pam_ref.pam_mul_ref(a, b)
    bad = np.flatnonzero(c != want)
    assert bad.size == 0, f"{bad.size} products differ, first at batch entry {bad[0]}"


@pytest.mark.parametrize("tile,kg,batch", [((64, 64), 1, 1), ((128, 64), 1, 2), ((64, 64), 4, 3)])
def test_whole_and_split_tiles_match_their_plans(tile, kg, batch):
    # Under a plan with whole-K tiles beside split ones, every whole tile is
    # bit for bit the unsplit plan's and every split tile the split plan's
    # (same K slices, added in the same order).
    import torch
    bm, bn = tile
    m, n, k = 200, 130, 700
    note(f"whole / split tiles vs their plans tile={tile} kgroups={kg} batch={batch}")
    g = np.random.default_rng(74)
    a = to_dev(g.standard_normal((batch, m, k)).astype(np.float32))
    b = to_dev(g.standard_normal((batch, k, n)).astype(np.float32))
    tiles_m, tiles_n = -(-m // bm), -(-n // bn)
    total = batch * tiles_m * tiles_n
    whole = total // 2 + 1
    unsplit = pam.bmm(a, b, plan=(bm, bn, 1, kg))
    split = pam.bmm(a, b, plan=(bm, bn, 4, kg))
    mixed = pam.bmm(a, b, plan=(bm, bn, 4, kg, whole))
    assert not torch.equal(unsplit.view(torch.int32), split.view(torch.int32))
    for t in range(total):
        z, r = divmod(t, tiles_m * tiles_n)
        tm, tn = divmod(r, tiles_n)
        sl = (z, slice(tm * bm, (tm + 1) * bm), slice(tn * bn, (tn + 1) * bn))
        want = unsplit if t < whole else split
        assert torch.equal(mixed[sl].view(torch.int32), want[sl].view(torch.int32)), f"tile {t}"


@pytest.mark.parametrize("ta,tb", TRANS, ids=["NN", "NT", "TN", "TT"])
def test_small_and_large_launches_agree(ta, tb):
    # A product's result does not depend on the launch it is part of: the
    # first 80 products of a batch (480 work items, fewer than the resident
    # workgroups; the kernel built for two waves per SIMD) and the same
    # products among 120 (720 work items; built for three) are bit for bit
    # equal, NaN payloads aside (the two builds may add the operands of a
    # SPECIAL step's sum in either order, and a sum of two NaNs keeps one of
    # them), and the small batch matches the oracle.
    import torch
    m, n, k = 200, 130, 700
    plan = (128, 64, 1, 2)
    note(f"small vs large launch m={m} n={n} k={k} ta={ta} tb={tb} plan={plan}")
    a_shape = (120, k, m) if ta else (120, m, k)
    b_shape = (120, n, k) if tb else (120, k, n)
    a = make("zeros_tiny", a_shape, 91)
    b = make("normal", b_shape, 92)
    a[7] = make("specials", a_shape[1:], 93)
    da, db = to_dev(a), to_dev(b)
    small = pam.bmm(da[:80], db[:80], trans_a=ta, trans_b=tb, plan=plan)
    large = pam.bmm(da, db, trans_a=ta, trans_b=tb, plan=plan)
    same_nan = torch.isnan(small) == torch.isnan(large[:80])
    assert bool(same_nan.all())
    fin = ~torch.isnan(small)
    assert torch.equal(small[fin].view(torch.int32), large[:80][fin].view(torch.int32))
    got = small[:8].cpu().numpy()
    c_ref, s_ref = oracle_gemm(a[:8], b[:8], ta, tb, m, n, k, a_shape[2], b_shape[2], a[0].size, b[0].size,
                               batches=list(range(8)))
    check_gemm(got, c_ref, s_ref, k, f"small launch ta={ta} tb={tb}")


def test_k0_writes_zeros():
    import torch
    note("gemm K = 0")
    a = torch.empty((7, 0), device=device())
    b = torch.empty((0, 9), device=device())
    c = torch.full((7, 9), 5.0, device=device())
    pam.gemm(a, b, out=c)
    assert torch.all(c == 0)
    # batched, into a padded output: every product zero, the padding untouched
    a3 = torch.empty((4, 5, 0), device=device())
    b3 = torch.empty((4, 0, 6), device=device())
    c3_full = torch.full((4, 5, 8), float("nan"), device=device())
    pam.bmm(a3, b3, out=c3_full[:, :, :6])
    assert torch.all(c3_full[:, :, :6] == 0)
    assert torch.all(torch.isnan(c3_full[:, :, 6:]))


def test_deterministic():
    import torch
    note("gemm bitwise repeatable, split-K plan")
    g = np.random.default_rng(73)
    a = to_dev(g.standard_normal((1, 200, 900)).astype(np.float32))
    b = to_dev(g.standard_normal((1, 900, 120)).astype(np.float32))
    for plan in ((64, 64, 6), (64, 64, 3, 4), (64, 64, 3, 1, 2)):
        c1 = pam.bmm(a, b, plan=plan)
        c2 = pam.bmm(a, b, plan=plan)
        assert torch.equal(c1.view(torch.int32), c2.view(torch.int32))


def test_linear_layer_forms_with_torch_views():
    """Forward and both approximate-derivative products of one linear layer."""
    import torch
    note("linear layer fwd / dX / dW through pam.gemm")
    g = np.random.default_rng(74)
    x = g.standard_normal((257, 96)).astype(np.float32)
    w = (0.05 * g.standard_normal((130, 96))).astype(np.float32)
    dy = (1e-3 * g.standard_normal((257, 130))).astype(np.float32)
    dx_, dw_, ddy = to_dev(x), to_dev(w), to_dev(dy)
    y = pam.gemm(dx_, dw_, trans_b=True).cpu().numpy()
    dX = pam.gemm(ddy, dw_).cpu().numpy()
    dW = pam.gemm(ddy, dx_, trans_a=True).cpu().numpy()
    for got, (a, b, ta, tb), k in ((y, (x, w, False, True), 96), (dX, (dy, w, False, False), 130),
                                   (dW, (dy, x, True, False), 257)):
        c_ref, s_ref = pam_ref.pam_gemm_ref(a, b, ta, tb)
        check_gemm(got, c_ref, s_ref, k, f"linear ta={ta} tb={tb}")


def pow2_operands(shape, seed, decoy_frac):
    """Signed powers of two 2^-57..2^-55, 5% zeros, some denormals, and
    'decoys' +-2^-72 (exponent field 55) whose products with every other
    operand underflow (below 2^-126) and must add exactly nothing."""
    g = np.random.default_rng(seed)
    e = g.integers(-57, -54, size=shape)
    x = (np.where(g.random(shape) < 0.5, 1.0, -1.0) * np.ldexp(1.0, e)).astype(np.float32)
    r = g.random(shape)
    x[r < 0.05] = 0.0
    x[(r >= 0.05) & (r < 0.06)] = np.float32(1e-40)
    x[(r >= 0.06) & (r < 0.06 + decoy_frac)] = np.float32(-(2.0 ** -72))
    return x


@pytest.mark.parametrize("decoys", [(0.0, 0.0), (0.01, 0.0), (0.0, 0.01), (0.02, 0.02), (0.3, 0.3)],
                         ids=["none", "A", "B", "both", "dense"])
@pytest.mark.parametrize("plan", [(128, 128, 1), (128, 64, 2), (128, 64, 1, 2), (64, 64, 1), (64, 64, 1, 4),
                                  (64, 64, 2, 4)],
                         ids=lambda p: "x".join(map(str, p)))
@pytest.mark.parametrize("ta,tb", [(False, True), (True, False)], ids=["NT", "TN"])
def test_exact_sums_underflowing_products_add_nothing(decoys, plan, ta, tb):
    """Every non-underflowing term is +-2^-114..2^-110 and the K = 300 sums
    need at most 13 bits, so any summation order is exact in float32: the
    result must equal the oracle bit for bit.  A product that underflows
    (below 2^-126) is zero by definition; adding anything for it would show."""
    m, n, k = 150, 140, 300
    note(f"exact pow2 sums decoys={decoys} plan={plan} ta={ta} tb={tb}")
    a_op = pow2_operands((m, k), 81, decoys[0])
    b_op = pow2_operands((k, n), 82, decoys[1])
    a = np.ascontiguousarray(a_op.T) if ta else a_op
    b = np.ascontiguousarray(b_op.T) if tb else b_op
    got = pam.bmm(to_dev(a[None]), to_dev(b[None]), trans_a=ta, trans_b=tb, plan=plan).cpu().numpy()[0]
    c_ref, _ = pam_ref.pam_gemm_ref(a, b, ta, tb)
    want = c_ref.astype(np.float32)
    assert np.array_equal(want.astype(np.float64), c_ref), "test data does not give exact float32 sums"
    bad = np.nonzero(got.view(np.uint32) != want.view(np.uint32))
    assert bad[0].size == 0, (f"{bad[0].size} outputs differ; first ({bad[0][0]}, {bad[1][0]}): "
                              f"got {got[bad][0]!r} want {want[bad][0]!r}")


def test_underflow_to_exact_zero_k1():
    """K = 1: products in the denormal range must come back as exact zeros."""
    note("K = 1 underflowing products")
    col = np.array([[2.0 ** -70], [1.5 * 2.0 ** -64], [-(2.0 ** -63)], [3.0]], dtype=np.float32)
    row = np.array([[2.0 ** -60, 1.25 * 2.0 ** -63, 2.0 ** -63, -(2.0 ** -100), 0.0]], dtype=np.float32)
    c = pam.gemm(to_dev(col), to_dev(row)).cpu().numpy()
    want = pam_ref.pam_mul_ref(np.repeat(col, 5, 1), np.repeat(row, 4, 0))
    assert np.array_equal(c, want), (c, want)
    assert np.all((c == 0) | (np.abs(c) >= 2.0 ** -126)), "a denormal value reached the output"


SEGMENT_MIXES = [(0.0, np.inf), (-0.0, np.nan), (np.float32(3e-41), -np.inf), (np.float32(1.2e-38), 2.0 ** 70),
                 (np.float32(-1.5e-38), np.float32(-(2.0 ** 65)))]


@pytest.mark.parametrize("plan", [(128, 128, 1), (128, 64, 1, 2), (64, 64, 1, 4)], ids=lambda p: "x".join(map(str, p)))
@pytest.mark.parametrize("ta,tb", TRANS, ids=["NN", "NT", "TN", "TT"])
@pytest.mark.parametrize("operand", ["A", "B"])
def test_special_beside_low_in_one_segment(operand, ta, tb, plan):
    # One group of four elements consecutive in memory (one staged segment)
    # holds a value below the S1 range next to a SPECIAL one, in one chunk of
    # one tile, all else normal: the chunk must take the SPECIAL path (the
    # special value must not hide behind the low one, nor the low one behind
    # the special) and the other chunks and tiles their own paths.
    m, n, k = 150, 140, 96
    for case, (low, special) in enumerate(SEGMENT_MIXES):
        a_shape = (k, m) if ta else (m, k)
        b_shape = (n, k) if tb else (k, n)
        g = np.random.default_rng(500 + case)
        a = g.standard_normal(a_shape).astype(np.float32)
        b = g.standard_normal(b_shape).astype(np.float32)
        x = a if operand == "A" else b
        r = int(g.integers(0, x.shape[0]))
        c0 = 4 * int(g.integers(0, x.shape[1] // 4))
        x[r, c0 + case % 4] = low
        x[r, c0 + (case + 2) % 4] = special
        note(f"segment mix {case} operand={operand} ta={ta} tb={tb} plan={plan} at ({r}, {c0})")
        c = pam.bmm(to_dev(a)[None], to_dev(b)[None], trans_a=ta, trans_b=tb, plan=plan)
        c_ref, s_ref = oracle_gemm(a.ravel(), b.ravel(), ta, tb, m, n, k, a.shape[1], b.shape[1], batches=[0])
        check_gemm(c.cpu().numpy(), c_ref, s_ref, k, f"segment mix {case} {operand} ta={ta} tb={tb} {plan}")


@pytest.mark.parametrize("where", ["first", "second", "both", "B"])
@pytest.mark.parametrize("plan", [(128, 128, 1), (128, 64, 1), (128, 64, 1, 2), (64, 64, 1), (64, 64, 1, 4),
                                  (128, 128, 3, 1, 2)], ids=lambda p: "x".join(map(str, p)))
@pytest.mark.parametrize("ta,tb", TRANS, ids=["NN", "NT", "TN", "TT"])
def test_low_values_in_one_half_of_the_tile_rows(where, plan, ta, tb):
    # Zeros, denormals and tiny normals only in the rows of op(A) that lie in
    # the first (second) half of their tile's rows, in both halves, or only
    # in B.  A k step then needs the zero / underflow handling for the rows
    # of one half and not for the other.  Two-mantissa-bit operands whose
    # sums are exact in any order: equal to the oracle bit for bit.
    import pam_workloads as wl
    m, n, k = 150, 140, 200
    tm = plan[0]
    note(f"low values in {where} rows plan={plan} ta={ta} tb={tb}")
    a_op = wl.exact_sum_values((m, k), 901, 0.0, 0.0)
    b_op = wl.exact_sum_values((k, n), 902, 0.0, 0.0)
    g = np.random.default_rng(903)
    low = wl.exact_sum_values((m + k, max(n, k)), 904, 0.5, 0.5)      # zeros, denormals, tiny normals
    if where == "B":
        hit = g.random((k, n)) < 0.01
        b_op[hit] = low[:k, :n][hit]
    else:
        half = (np.arange(m) % tm) >= tm // 2
        rows = {"first": ~half, "second": half, "both": np.ones(m, bool)}[where]
        hit = (g.random((m, k)) < 0.03) & rows[:, None]
        a_op[hit] = low[:m, :k][hit]
    a = np.ascontiguousarray(a_op.T) if ta else a_op
    b = np.ascontiguousarray(b_op.T) if tb else b_op
    got = pam.bmm(to_dev(a[None]), to_dev(b[None]), trans_a=ta, trans_b=tb, plan=plan).cpu().numpy()[0]
    c_ref, _ = pam_ref.pam_gemm_ref(a, b, ta, tb)
    assert np.array_equal(c_ref.astype(np.float32).astype(np.float64), c_ref), "test data does not sum exactly"
    bad = np.nonzero(got.astype(np.float64) != c_ref)
    assert bad[0].size == 0, (f"{bad[0].size} outputs differ; first ({bad[0][0]}, {bad[1][0]}): "
                              f"got {got[bad][0]!r} want {c_ref[bad][0]!r}")
