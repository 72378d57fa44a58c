"""Full-size workloads, in the launch configuration the benchmark times.

Every product of every workload runs at its real shape with the automatic
plan.  The oracle checks sampled outputs (whole rows, plus whole columns for
the long-K weight-gradient products, and whole batch entries for attention);
properties that hold at any size (no NaN/inf on finite inputs, deterministic
repeat) are checked on the full output.
"""
import numpy as np
import pytest

import pam_workloads as wl
import paper_2305_17190_amd as pam
from gpu_util import check_gemm, note, oracle_gemm, to_dev

pytestmark = pytest.mark.gpu

_cache = {}


def dev_inputs(w):
    if w not in _cache:
        _cache.clear()
        host = wl.workload_inputs(w)
        _cache[w] = (host, {k: to_dev(v) for k, v in host.items()})
    return _cache[w]


def run_form(form, dt):
    import torch
    A, B = dt[form.a], dt[form.b]
    if form.batch > 1:
        return pam.bmm(A, B, trans_a=form.trans_a, trans_b=form.trans_b)
    return pam.gemm(A, B, trans_a=form.trans_a, trans_b=form.trans_b)


def sample(n, count, seed):
    g = np.random.default_rng(seed)
    idx = np.sort(g.choice(n, size=min(n, count), replace=False))
    # always include both ends (ragged last tile)
    return np.unique(np.concatenate([idx, [0, n - 1]]))


CASES = [(w, f.name) for w in (1, 2, 3, 4, 5) for f in wl.WORKLOADS[w]["forms"]]


@pytest.mark.parametrize("w,name", CASES, ids=[f"w{w}-{n}" for w, n in CASES])
def test_workload_form(w, name):
    import torch
    form = next(f for f in wl.WORKLOADS[w]["forms"] if f.name == name)
    note(f"workload {w} {name}: m={form.m} n={form.n} k={form.k} batch={form.batch} plan={pam.plan(form.m, form.n, form.k, form.batch)}")
    host, dt = dev_inputs(w)
    c = run_form(form, dt)
    torch.cuda.synchronize()
    assert torch.isfinite(c).all().item(), "non-finite output on finite inputs"
    c2 = run_form(form, dt)
    assert torch.equal(c.view(torch.int32), c2.view(torch.int32)), "not bitwise repeatable"
    a_buf, b_buf = host[form.a], host[form.b]
    if form.batch > 1:
        bats = sample(form.batch, 3, 7)
        c_ref, s_ref = oracle_gemm(a_buf, b_buf, form.trans_a, form.trans_b, form.m, form.n, form.k, form.lda,
                                   form.ldb, form.stride_a, form.stride_b, batches=bats)
        got = c.cpu().numpy()[bats]
        check_gemm(got, c_ref, s_ref, form.k, f"w{w} {name} batches {list(bats)}")
        return
    big = form.m * form.n * form.k > 2e10
    rows = sample(form.m, 24 if big else 96, 1)
    c_ref, s_ref = oracle_gemm(a_buf, b_buf, form.trans_a, form.trans_b, form.m, form.n, form.k, form.lda,
                               form.ldb, rows=rows)
    got = c.cpu().numpy()
    check_gemm(got[rows], c_ref[0], s_ref[0], form.k, f"w{w} {name} rows")
    cols = sample(form.n, 8 if big else 32, 2)
    c_ref, s_ref = oracle_gemm(a_buf, b_buf, form.trans_a, form.trans_b, form.m, form.n, form.k, form.lda,
                               form.ldb, cols=cols)
    check_gemm(got[:, cols], c_ref[0], s_ref[0], form.k, f"w{w} {name} cols")
