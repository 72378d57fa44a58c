"""Properties of the library's plan choice over random sizes (host logic, no
GPU): a valid tile shape and split count, K slices of at least four chunks,
hybrid plans whose whole-K tiles fill whole rounds of resident workgroups and
split only the last one (or one and a half), and a workspace size that
matches the plan."""
import ctypes

from hypothesis import given, settings, strategies as st

import paper_2305_17190_amd as pam

# Resident workgroups of each tile shape on the 256 compute units.
SLOTS = {(128, 128, 1): 3 * 256, (128, 64, 1): 4 * 256, (128, 64, 2): 2 * 256, (64, 64, 1): 8 * 256,
         (64, 64, 4): 2 * 256}


@settings(max_examples=3000, deadline=None)
@given(m=st.integers(1, 70000), n=st.integers(1, 70000), k=st.integers(1, 200000),
       batch=st.sampled_from([1, 1, 1, 2, 3, 8, 64, 256, 1000]))
def test_plans_are_valid(m, n, k, batch):
    if m * n * batch > (1 << 34):         # beyond any output this GPU can hold
        return
    tm, tn, splits, kg, whole = pam.plan(m, n, k, batch)
    assert (tm, tn, kg) in SLOTS
    assert 1 <= splits <= 64
    tiles = -(-m // tm) * -(-n // tn) * batch
    if splits > 1:
        per = -(-k // splits)
        assert per >= 4 * 16 * kg or splits == 1, (per, kg)
        assert 0 <= whole < tiles
        if whole:
            slots = SLOTS[(tm, tn, kg)]
            assert whole % slots == 0
            assert tiles - whole in (tiles % slots, tiles % slots + slots)
    else:
        assert whole == 0
    size = ctypes.c_size_t()
    assert pam.load().pam_gemm_workspace_size(m, n, k, batch, ctypes.byref(size)) == 0
    split_tiles = 0 if splits == 1 else (tiles - whole if whole else tiles)
    if splits > 1 and not whole:
        # plain split-K: the workspace holds one launch's worth of matrices
        per_launch = max(1, 16777215 // ((tiles // batch) * splits))
        split_tiles = min(batch, per_launch) * (tiles // batch)
    assert size.value == splits * split_tiles * tm * tn * 4
