"""The element-wise full-size parity checker, run on the CPU against the oracle's own outputs.

It must pass on exact outputs and fail when one element of one tensor is off by more than the
bf16 tolerance: a planted error in one key of the most-shared node's first tile (dK), in one row
of a consumer of that node (O), and in a leaf's last query tile (dQ); and, through the complete
slices, in a key in the middle of the most-shared node (dK, dV) and in a middle row of the
checked branch (dQ), which the first and last tiles alone do not cover.
"""
import numpy as np
import pytest

from paper_2608_25683_amd import workloads as W
import parity_helpers as H


@pytest.fixture(scope="module")
def case():
    wl = W.custom([-1, 0, 0, 1, 1], [200, 70, 150, 40, 9], [3, 4, 2], hq=8, hkv=2, d=64, dtype="bf16", seed=5,
                  block_policy=lambda L: W.blocks_fixed(L, 32))
    return wl, H.run_oracle(wl)


def test_exact_outputs_pass(case):
    wl, ref = case
    res = H.check_full_size(wl, ref, workers=2)
    assert res["shared_node"] == 0 and res["o_rows"] >= wl.tree.num_rows   # every row consumes the root
    for k in ("O", "LSE", "dQ", "dK", "dV"):
        assert res[k][0] < 1e-5, (k, res[k])


@pytest.mark.parametrize("which", ["dK", "O", "dQ"])
def test_planted_error_fails(case, which):
    wl, ref = case
    out = [x.copy() for x in ref]
    t = wl.tree
    if which == "dK":
        out[3][t.row_slots()[3], 1, 7] += 0.05          # key row 3 of the root, kv head 1
    elif which == "O":
        out[0][t.row_off[4] + 2, 5, 0] += 0.05          # a row of node 4, query head 5
    else:
        out[2][t.row_off[2] + t.seg_len[2] - 1, 0, 3] += 0.05   # last row of the longest leaf
    with pytest.raises(AssertionError, match=which):
        H.check_full_size(wl, tuple(out), workers=2)


# the complete slices (kv head 0: every key of the most-shared node and of the leaf, and dQ of
# every row of one branch) catch errors that the first and last tiles do not cover
@pytest.fixture(scope="module")
def case_long():
    wl = W.custom([-1, 0, 0], [400, 300, 150], [1, 2], hq=4, hkv=2, d=64, dtype="bf16", seed=6,
                  block_policy=lambda L: W.blocks_fixed(L, 32))
    return wl, H.run_oracle(wl)


def test_complete_slices_pass(case_long):
    wl, ref = case_long
    res = H.check_full_size(wl, ref, workers=2)
    assert res["keys complete"] == 400 + 300 and res["dq_rows complete"] == 300 and res["branch"] == 1
    for k in ("dK complete", "dV complete", "dQ complete"):
        assert res[k][0] < 1e-5, (k, res[k])


@pytest.mark.parametrize("which", ["dK", "dV", "dQ"])
def test_planted_error_in_a_middle_tile_fails(case_long, which):
    wl, ref = case_long
    out = [x.copy() for x in ref]
    t = wl.tree
    if which in ("dK", "dV"):
        out[3 if which == "dK" else 4][t.row_slots()[200], 0, 11] += 0.05   # root key 200, kv head 0
    else:
        out[2][t.row_off[1] + 150, 1, 5] += 0.05                            # middle row of the branch
    with pytest.raises(AssertionError, match=which):
        H.check_full_size(wl, tuple(out), workers=2)
    res = H.check_full_size(wl, tuple(out), workers=2, complete=False)   # the tiles alone miss it
    assert res[which][0] < 1e-5
