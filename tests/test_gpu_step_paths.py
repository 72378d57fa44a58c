"""The matrix product's per-wave choice of k-step path.

Within each LDS chunk a wave takes the k steps whose operands (the A rows it
owns, the B columns of the tile) all have exponent fields in [64, 190] on
the two-op integer-add path, in pairs with the next step's operands read
ahead and one step alone first when their count is odd; then the steps with
zeros or denormals (add + fma), then those with tiny normals (add, mul,
add).  Zeros and tiny values planted at chosen (row, k) places of A give the
waves of a 128 x 128 tile every count of two-op steps from 0 to 16 across
the chunks (and other mixes under the other tile shapes); columns of B that
are zero or tiny at some k move that step off the two-op path for every
wave.  Each product is compared with the oracle within the GEMM tolerance.
"""
import numpy as np
import pytest

import paper_2305_17190_amd as pam
from gpu_util import check_gemm, note, oracle_gemm, to_dev

pytestmark = pytest.mark.gpu

CHUNKS = 17
M, N, K = 256, 128, 16 * CHUNKS
TINY = np.float32(1.5e-38)   # normal, exponent field 1: its products underflow


def planted_operands(seed):
    rng = np.random.default_rng(seed)
    a = rng.standard_normal((M, K)).astype(np.float32)
    b = rng.standard_normal((K, N)).astype(np.float32)
    for c in range(CHUNKS):
        for w in range(4):
            # A 128-row tile's wave w owns rows 16w..16w+15 and 64+16w..64+16w+15
            off = (c + 5 * w) % CHUNKS            # this chunk's k steps wave w takes off the two-op path
            for j, kk in enumerate(rng.permutation(16)[:off] + 16 * c):
                for tile_row in range(M // 128):
                    row = tile_row * 128 + (64 if j % 2 else 0) + 16 * w + int(rng.integers(0, 16))
                    a[row, kk] = np.float32(0.0) if j % 3 else (TINY if j % 2 else -TINY)
    # B: in chunk 3 one zero column entry, in chunk 9 one tiny one (every wave's step)
    b[16 * 3 + 5, 17] = 0.0
    b[16 * 9 + 11, 100] = TINY
    return a, b


@pytest.mark.parametrize("plan", [(128, 128, 1, 1, 0), (128, 64, 1, 1, 0), (128, 64, 1, 2, 0), (64, 64, 1, 1, 0),
                                  (64, 64, 1, 4, 0)])
@pytest.mark.parametrize("ta,tb", [(False, False), (False, True), (True, False)])
def test_every_two_op_step_count(ta, tb, plan):
    a, b = planted_operands(31)
    note(f"step paths ta={ta} tb={tb} plan={plan} m={M} n={N} k={K}")
    a_buf = np.ascontiguousarray(a.T if ta else a)
    b_buf = np.ascontiguousarray(b.T if tb else b)
    c = pam.bmm(to_dev(a_buf)[None], to_dev(b_buf)[None], trans_a=ta, trans_b=tb, plan=plan)
    c_ref, s_ref = oracle_gemm(a_buf.ravel(), b_buf.ravel(), ta, tb, M, N, K, a_buf.shape[1], b_buf.shape[1],
                               batches=[0])
    check_gemm(c.cpu().numpy(), c_ref, s_ref, K, f"step paths ta={ta} tb={tb} plan={plan}")

