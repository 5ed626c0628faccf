"""Cross-call prefix reuse on the host (Sec. 4.1.1 inter-batch sharing, Sec. 4.1.2 self-sequence
sharing): a forest processed over several calls, where a later call reads the K/V of nodes an
earlier call computed (external nodes: row_off = -1, no query rows) and adds its share of their
dK/dV to what the earlier calls left.

Checked through the C ABI without a GPU: descriptor rules for external nodes, and the plans of
the calls together cover every visible (query, key) pair of the whole forest exactly once -- in
the forward and dQ items of the call that holds the query, and in the dK/dV items, which are
marked to accumulate exactly when their keys belong to an external node.
"""
import numpy as np
import pytest

from paper_2608_25683_amd import workloads as W

P = pytest.importorskip("paper_2608_25683_amd.psattn")


def _forest():
    # root(150) -> a(70) -> c(40); root -> b(33); root -> d(9); samples end at c, b, d
    return W.custom([-1, 0, 0, 1, 0], [150, 70, 33, 40, 9], [3, 2, 4], hq=8, hkv=2, d=128, tensors=False,
                    block_policy=lambda L: W.blocks_fixed(L, 32), seed=3)


def _forest_pairs(tree):
    """(row, key row) pairs of the forest's mask."""
    off = tree.node_offsets()
    pairs = set()
    for n in range(tree.num_nodes):
        prow = np.concatenate([np.arange(tree.row_off[m], tree.row_off[m] + tree.seg_len[m]) for m in tree.path(n)])
        for a in range(int(tree.seg_len[n])):
            for k in prow[: int(off[n]) + a + 1]:
                pairs.add((int(tree.row_off[n]) + a, int(k)))
    return pairs


def _call_cover(forest, call, rows, t):
    """Forest (row, key) pairs covered by one call's forward and dK/dV items, with the dK/dV
    items' accumulate flags; asserts each pair once per head within the call."""
    slot_to_row = {int(s): r for r, s in enumerate(forest.tree.row_slots())}
    q_list, kv_list = t.plan_array("q_list"), t.plan_array("kv_list")
    row_pos = t.plan_array("row_pos")
    fwd, bkv = t.plan_array("fwd_items"), t.plan_array("bkv_items")
    hc = t.info["head_chunk"]
    f_cover, b_cover, acc_keys, write_keys = {}, {}, set(), set()
    for q_off, nq, kv_off, nkv, kv_pos0, head0, part, nfull in fwd:
        keys = [slot_to_row[int(s)] for s in kv_list[kv_off:kv_off + nkv]]
        for r in q_list[q_off:q_off + nq]:
            for j, k in enumerate(keys):
                if kv_pos0 + j <= row_pos[r]:
                    for h in range(head0, head0 + hc):
                        key = (h, int(rows[r]), k)
                        f_cover[key] = f_cover.get(key, 0) + 1
    for kv_off, nk, kv_pos0, q_off, nq, hk, part, mask_lo, mask_hi, acc in bkv:
        keys = [slot_to_row[int(s)] for s in kv_list[kv_off:kv_off + nk]]
        (acc_keys if acc else write_keys).update(keys)
        for r in q_list[q_off:q_off + nq]:
            for j, k in enumerate(keys):
                if row_pos[r] >= kv_pos0 + j:
                    key = (hk, int(rows[r]), k)
                    b_cover[key] = b_cover.get(key, 0) + 1
    assert all(v == 1 for v in f_cover.values()) and all(v == 1 for v in b_cover.values())
    return f_cover, b_cover, acc_keys, write_keys


@pytest.mark.parametrize("split", [([0], [1, 2]), ([1], [0, 2]), ([2], [0, 1])])
def test_two_calls_cover_the_forest_once(split):
    forest = _forest()
    t = forest.tree
    ends_a = [int(t.sample_end[s]) for s in split[0]]
    ends_b = [int(t.sample_end[s]) for s in split[1]]
    call_a, rows_a = W.call_subset(forest, ends_a)
    done = set(int(n) for n in np.nonzero(np.isin(np.arange(t.num_nodes), [m for e in ends_a for m in t.path(e)]))[0])
    call_b, rows_b = W.call_subset(forest, ends_b, external=done)
    ta = P.Tree.from_workload(call_a)
    tb = P.Tree.from_workload(call_b)
    assert ta.num_rows == len(rows_a) and tb.num_rows == len(rows_b)
    assert len(set(rows_a) | set(rows_b)) == t.num_rows and not set(rows_a) & set(rows_b)
    pairs = _forest_pairs(t)
    fa, ba, acc_a, wr_a = _call_cover(forest, call_a, rows_a, ta)
    fb, bb, acc_b, wr_b = _call_cover(forest, call_b, rows_b, tb)
    # forward/dQ: each visible pair once per query head over both calls
    assert not set(fa) & set(fb)
    assert len(fa) + len(fb) == len(pairs) * forest.hq
    # dK/dV: each visible pair once per kv head over both calls
    assert not set(ba) & set(bb)
    assert len(ba) + len(bb) == len(pairs) * forest.hkv
    # the first call writes every key it covers; the second accumulates exactly into the cached
    # (external) keys, which the first call wrote
    assert not acc_a
    ext_rows = {r for n in done for r in range(int(t.row_off[n]), int(t.row_off[n] + t.seg_len[n]))}
    assert acc_b == ext_rows & (acc_b | wr_b) and acc_b <= wr_a and not (wr_b & ext_rows)
    # padding zeroed only inside the call's own (internal) blocks
    for call, tr in ((call_a, ta), (call_b, tb)):
        own = set()
        c = call.tree
        for n in range(c.num_nodes):
            if c.row_off[n] >= 0:
                for b in range(int(c.blk_ptr[n]), int(c.blk_ptr[n + 1])):
                    own |= set(range(int(c.blk_base[b]) + int(c.blk_len[b]), int(c.blk_base[b]) + int(c.blk_cap[b])))
        assert set(tr.plan_array("pad_slots").tolist()) == own


def test_chunked_sequence_calls():
    # one 420-token sequence as a chain of three chunks, one call per chunk
    wl = W.custom([-1, 0, 1], [160, 130, 130], [2], hq=4, hkv=1, d=64, tensors=False, block_policy=W.blocks_greedy,
                  seed=4)
    covered = {}
    for c in range(3):
        call, rows = W.call_subset(wl, [c], external=range(c))
        tr = P.Tree.from_workload(call, opts={"bwd_q_chunk": 64})
        assert tr.info["unshared_tokens"] == (130 if c else 160)
        _, b, acc, wr = _call_cover(wl, call, rows, tr)
        for k in b:
            assert k not in covered
            covered[k] = c
        assert acc == set(range(0, int(wl.tree.row_off[c]))) if c else not acc
    assert len(covered) == len(_forest_pairs(wl.tree)) * wl.hkv


@pytest.mark.parametrize("mutate", ["internal_under_external_ok", "external_under_internal", "sample_at_external",
                                    "all_external"])
def test_external_node_rules(mutate):
    forest = _forest()
    t = forest.tree
    call, _ = W.call_subset(forest, [int(t.sample_end[0])], external=[0])   # root cached
    d = dict(parent=call.tree.parent, seg_len=call.tree.seg_len, row_off=call.tree.row_off.copy(),
             blk_ptr=call.tree.blk_ptr, blk_base=call.tree.blk_base, blk_cap=call.tree.blk_cap,
             blk_len=call.tree.blk_len, blk_pos=call.tree.blk_pos, pool_slots=call.tree.pool_slots,
             sample_end=call.tree.sample_end.copy(), hq=8, hkv=2, head_dim=128, softmax_scale=0.088)
    if mutate == "internal_under_external_ok":
        assert P.Tree(**d).num_rows == 110
        return
    if mutate == "external_under_internal":       # root internal, its child external
        d["row_off"] = np.array([0, -1, 150], dtype=np.int64)
    elif mutate == "sample_at_external":
        d["sample_end"] = np.array([0], dtype=np.int32)
    else:
        d["row_off"] = np.full(3, -1, dtype=np.int64)
    with pytest.raises(P.PsattnError) as e:
        P.Tree(**d)
    assert e.value.name == "PSATTN_E_INVALID_TREE"
