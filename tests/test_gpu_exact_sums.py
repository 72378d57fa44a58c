"""Bit-exact parity of the benchmark's own products at full size.

Every product of workloads w2-w5 runs at its real shape under the plan the
library picks for it -- w5's hybrid plans (whole-K tiles, then the last
round's tiles in K slices), the 61-way split of w2's dW, the 32-way splits of
w3's weight gradients, w4's batched products -- and, for the long-K weight
gradients, also under the plan of the entry points without a workspace.  The
operands are signed values with two mantissa bits and exponents in [-6, -3]
(PAM still differs from multiplication on them), with planted zeros,
denormals and tiny normals that drive the kernels' zero and underflow step
paths.  Every sum of such PAM terms is exact in float32 in any order, so the
GPU must equal the oracle bit for bit (up to the sign of an exact zero): a
dropped, repeated or misplaced LDS chunk or K slice shows.  Sampled outputs:
rows from the whole-K tiles and from the split tiles, and whole columns.

The Sec. 2.2 underflow rule at its rounding tie: 0x1FFFFFFF .^ 0x20000000 sums
to 0x007FFFFF, a signed zero, while the product the underflow step forms is
exactly 2^-126 - 2^-150; every tile shape, both operand orders.
"""
import numpy as np
import pytest

import pam_workloads as wl
import paper_2305_17190_amd as pam
from gpu_util import device, note, oracle_gemm, to_dev

pytestmark = pytest.mark.gpu

_cache = {}


def operand_shape(form, which):
    if form.batch > 1:
        rows, cols = ((form.k, form.m) if form.trans_a else (form.m, form.k)) if which == "a" else \
            ((form.n, form.k) if form.trans_b else (form.k, form.n))
        return (form.batch, rows, cols)
    if which == "a":
        return (form.k, form.m) if form.trans_a else (form.m, form.k)
    return (form.n, form.k) if form.trans_b else (form.k, form.n)


def exact_inputs(w):
    if w not in _cache:
        _cache.clear()
        shapes = {}
        for f in wl.WORKLOADS[w]["forms"]:
            shapes[f.a] = operand_shape(f, "a")
            shapes[f.b] = operand_shape(f, "b")
        host = {name: wl.exact_sum_values(shape, 7000 * w + i) for i, (name, shape) in enumerate(sorted(shapes.items()))}
        _cache[w] = (host, {k: to_dev(v) for k, v in host.items()})
    return _cache[w]


def split_rows(form, plan):
    """Rows of op(A) that lie in K-split tiles under `plan` (batch 1)."""
    tm, tn, splits, kg, whole = plan
    if splits == 1:
        return np.zeros(0, np.int64)
    tiles_n = -(-form.n // tn)
    tiles = -(-form.m // tm) * tiles_n
    first = whole if whole else 0
    if first >= tiles:
        return np.zeros(0, np.int64)
    row0 = (first // tiles_n) * tm
    return np.arange(row0, form.m)


def pick(idx, count, seed):
    g = np.random.default_rng(seed)
    if idx.size <= count:
        return idx
    return np.sort(g.choice(idx, size=count, replace=False))


def run(form, dt, entry):
    import torch
    A, B = dt[form.a], dt[form.b]
    if form.batch > 1:
        return pam.bmm(A, B, trans_a=form.trans_a, trans_b=form.trans_b)
    if entry == "workspace":
        return pam.gemm(A, B, trans_a=form.trans_a, trans_b=form.trans_b)
    # the C entry point without a workspace, through its own plan
    lib = pam.load()
    c = torch.empty((form.m, form.n), device=device())
    st = lib.pam_gemm(1 if form.trans_a else 0, 1 if form.trans_b else 0, form.m, form.n, form.k, A.data_ptr(),
                      form.lda, B.data_ptr(), form.ldb, c.data_ptr(), form.n,
                      torch.cuda.current_stream().cuda_stream)
    assert st == 0
    return c


CASES = [(w, f.name, "workspace") for w in (2, 3, 4, 5) for f in wl.WORKLOADS[w]["forms"]]
CASES += [(2, "dW", "none"), (3, "dW2", "none"), (5, "dW", "none"), (5, "fwd", "none")]


@pytest.mark.parametrize("w,name,entry", CASES, ids=[f"w{w}-{n}-{e}" for w, n, e in CASES])
def test_full_shape_exact_sums(w, name, entry):
    import torch
    form = next(f for f in wl.WORKLOADS[w]["forms"] if f.name == name)
    plan = pam.plan(form.m, form.n, form.k, form.batch, max_workspace_bytes=None if entry == "workspace" else 0)
    note(f"exact sums w{w} {name} ({entry}): m={form.m} n={form.n} k={form.k} batch={form.batch} plan={plan}")
    host, dt = exact_inputs(w)
    c = run(form, dt, entry)
    torch.cuda.synchronize()
    got = c.cpu().numpy().astype(np.float64)
    a_buf, b_buf = host[form.a], host[form.b]
    if form.batch > 1:
        bats = np.unique(np.concatenate([pick(np.arange(form.batch), 3, 11), [form.batch - 1]]))
        c_ref, s_ref = oracle_gemm(a_buf, b_buf, form.trans_a, form.trans_b, form.m, form.n, form.k, form.lda,
                                   form.ldb, form.stride_a, form.stride_b, batches=bats)
        assert np.all(s_ref > 0)
        assert np.array_equal(got[bats], c_ref), f"w{w} {name}: batches {list(bats)} differ"
        return
    big = form.m * form.n * form.k > 2e10
    count = 16 if big else 48
    split = split_rows(form, plan)
    whole = np.setdiff1d(np.arange(form.m), split)
    rows = np.unique(np.concatenate([pick(whole, count, 1), pick(split, count, 2), [0, form.m - 1]]))
    c_ref, s_ref = oracle_gemm(a_buf, b_buf, form.trans_a, form.trans_b, form.m, form.n, form.k, form.lda,
                               form.ldb, rows=rows)
    bad = got[rows] != c_ref[0]
    assert not bad.any(), (f"w{w} {name}: {int(bad.sum())} of {bad.size} sampled outputs differ "
                           f"(split-tile rows sampled: {int(np.isin(rows, split).sum())})")
    cols = np.unique(np.concatenate([pick(np.arange(form.n), 6 if big else 16, 3), [form.n - 1]]))
    c_ref, s_ref = oracle_gemm(a_buf, b_buf, form.trans_a, form.trans_b, form.m, form.n, form.k, form.lda,
                               form.ldb, cols=cols)
    bad = got[:, cols] != c_ref[0]
    assert not bad.any(), f"w{w} {name}: {int(bad.sum())} of {bad.size} sampled column outputs differ"


TILES = [(128, 128, 1, 1), (128, 64, 1, 1), (128, 64, 1, 2), (64, 64, 1, 1), (64, 64, 1, 4)]
TIE_LO = np.uint32(0x1FFFFFFF).view(np.float32)     # exponent field 63, mantissa all ones
TIE_HI = np.uint32(0x20000000).view(np.float32)     # exponent field 64, mantissa zero


@pytest.mark.parametrize("tile", TILES, ids=lambda t: "x".join(map(str, t)))
@pytest.mark.parametrize("order", ["tiny_a", "tiny_b"])
def test_underflow_tie_is_zero(tile, order):
    """One k step pairs 0x1FFFFFFF with 0x20000000 (either side) in every
    output, with opposite signs in half of them; the other steps hold
    exact-sum values.  The tie pair adds nothing (R4), so C equals the
    oracle bit for bit."""
    import torch
    from oracle import pam_ref
    note(f"underflow tie, tile {tile}, {order}")
    assert pam_ref.pam_mul_ref(TIE_LO, TIE_HI).view(np.uint32) == 0
    m, n, k = 150, 90, 40
    a = wl.exact_sum_values((m, k), 61, 0.0, 0.0)
    b = wl.exact_sum_values((k, n), 62, 0.0, 0.0)
    g = np.random.default_rng(63)
    sa = np.where(g.random(m) < 0.5, -1.0, 1.0).astype(np.float32)
    sb = np.where(g.random(n) < 0.5, -1.0, 1.0).astype(np.float32)
    lo, hi = (TIE_LO, TIE_HI) if order == "tiny_a" else (TIE_HI, TIE_LO)
    a[:, 17] = sa * lo
    b[17, :] = sb * hi
    tm, tn, splits, kg = tile
    c = pam.bmm(to_dev(a[None]), to_dev(b[None]), plan=(tm, tn, splits, kg, 0)).cpu().numpy()[0]
    c_ref, _ = pam_ref.pam_gemm_ref(a, b)
    assert np.array_equal(c.astype(np.float64), c_ref)
    # K = 1: the tie pair alone gives zeros
    c1 = pam.bmm(to_dev(a[None, :, 17:18]), to_dev(b[None, 17:18, :]), plan=(tm, tn, 1, kg, 0)).cpu().numpy()[0]
    assert np.all(c1 == 0.0), f"{int((c1 != 0).sum())} outputs nonzero, e.g. {c1[c1 != 0][:3]}"
