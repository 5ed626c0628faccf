"""The adaptive KV cache manager (Sec. 5.1 adaptive block allocation, Sec. 5.2 dynamic block
caching, farthest-next-use eviction), through the C ABI on the host.

Pinned to the paper's two worked examples (tests/golden/paper_structure_examples.json): the
28 + 4 + 4 adaptive blocks of Fig. "Block_Management", and the reference counts 4/3/1 with the
third block freed after sample a of Fig. "Generation_Prefix_Tree".  Every call's descriptor is
accepted by psattn_tree_create; eviction follows the farthest next use; a synthetic peak-memory
comparison (dynamic caching against keeping every block, adaptive blocks against fixed pages).
"""
import json
import pathlib

import numpy as np
import pytest

from paper_2608_25683_amd import workloads as W

P = pytest.importorskip("paper_2608_25683_amd.psattn")
GOLDEN = json.loads((pathlib.Path(__file__).parent / "golden" / "paper_structure_examples.json").read_text())


def _tree_of(plan, c, hq=4, hkv=2, d=64):
    x = plan.call(c)
    return x, P.Tree(parent=x["parent"], seg_len=x["seg_len"], row_off=x["row_off"], blk_ptr=x["blk_ptr"],
                     blk_base=x["blk_base"], blk_cap=x["blk_cap"], blk_len=x["blk_len"], blk_pos=x["blk_pos"],
                     pool_slots=x["pool_slots"], sample_end=x["sample_end"], hq=hq, hkv=hkv, head_dim=d,
                     softmax_scale=0.125)


def test_adaptive_block_example():
    g = GOLDEN["adaptive_block_example"]
    ada = P.KVCachePlan(g["parent"], g["seg_len"], [1, 2], [0, 0], capacity=1000)
    assert ada.stats["peak_slots"] == g["adaptive"]["pool_slots"]            # 28 + 4 + 4
    x = ada.call(0)
    assert sorted(x["blk_len"].tolist()) == sorted(g["adaptive"]["blk_len"]) and np.all(x["blk_cap"] == x["blk_len"])
    fixed = P.KVCachePlan(g["parent"], g["seg_len"], [1, 2], [0, 0], capacity=1000, block_size=32)
    assert fixed.stats["peak_slots"] == g["fixed_32"]["pool_slots"]
    assert fixed.stats["peak_slots"] - sum(g["seg_len"]) == g["fixed_32"]["pad_slots"]


def test_dbc_example_reference_counts_and_release():
    g = GOLDEN["dbc_example"]
    # samples a, b, c, d in calls 0..3 (one micro-batch each)
    plan = P.KVCachePlan(g["parent"], g["seg_len_illustrative"], g["samples"], [0, 1, 2, 3], capacity=1000)
    freed = [[e[1] for e in plan.events(c, 1) if e[0] == "free"] for c in range(4)]
    # after sample a: root (read by abcd) and X (abc) stay, a's own block is freed
    assert freed[0] == [2]
    assert freed[1] == [3]
    assert sorted(freed[2]) == [1, 4]          # X's last reader is c
    assert sorted(freed[3]) == [0, 5]          # the root's last reader is d
    # the reference counts the release follows are the paper's 4/3/1
    t = P.Tree(parent=g["parent"], seg_len=g["seg_len_illustrative"],
               row_off=np.concatenate([[0], np.cumsum(g["seg_len_illustrative"])[:-1]]),
               blk_ptr=np.arange(7), blk_base=np.concatenate([[0], np.cumsum(g["seg_len_illustrative"])[:-1]]),
               blk_cap=g["seg_len_illustrative"], blk_len=g["seg_len_illustrative"],
               blk_pos=[0, 6, 10, 10, 10, 6], pool_slots=sum(g["seg_len_illustrative"]), sample_end=g["samples"],
               hq=4, hkv=2, head_dim=64, softmax_scale=0.125)
    assert t.refcounts().tolist() == g["refcounts"]
    # later calls read the root (and X) from the cache
    for c in range(1, 4):
        x = plan.call(c)
        ext = {int(n) for n, r in zip(x["node_ids"], x["row_off"]) if r < 0}
        assert 0 in ext and (1 in ext if c < 3 else True)


def test_every_call_descriptor_is_a_valid_tree():
    wl = W.make("c4", tensors=False)
    t = wl.tree
    calls = np.arange(len(t.sample_end)) // 8                                    # 8 micro-batches of 8 leaves
    plan = P.KVCachePlan(t.parent, t.seg_len, t.sample_end, calls, capacity=t.num_rows)
    computed = set()
    for c in range(plan.num_calls):
        x, tree = _tree_of(plan, c)
        ids = x["node_ids"]
        internal = {int(ids[i]) for i in range(len(ids)) if x["row_off"][i] >= 0}
        assert not internal & computed                                          # each node computed once
        assert {int(n) for n in ids} - internal <= computed                     # the rest from the cache
        computed |= internal
        assert tree.num_rows == sum(int(t.seg_len[n]) for n in internal)
        assert [e[1] for e in plan.events(c, 0) if e[0] == "alloc"] == sorted(internal)
    assert computed == set(range(t.num_nodes))
    assert plan.stats["final_slots"] == 0 and plan.stats["evictions"] == 0


def test_farthest_next_use_is_evicted():
    # three 100-token roots r0, r1, r2; reads: r0 | r1 | r2 | r0 | r1, room for two roots
    parent, seg = [-1, -1, -1], [100, 100, 100]
    plan = P.KVCachePlan(parent, seg, [0, 1, 2, 0, 1], [0, 1, 2, 3, 4], capacity=200)
    before2 = plan.events(2, 0)
    assert [e[:2] for e in before2] == [("evict", 1), ("alloc", 2)]              # r1 is next read at call 4
    assert plan.events(3, 0) == []                                               # r0 still cached
    # r2 (after call 2) and r0 (after call 3) reached reference count 0 and were freed: r1 comes
    # back without another eviction
    assert [e[:2] for e in plan.events(4, 0)] == [("refill", 1)]
    x = plan.call(4)
    assert x["row_off"].tolist() == [-1]                                         # read from the refilled block
    assert plan.stats["evictions"] == 1 and plan.stats["refilled_tokens"] == 100
    assert plan.stats["peak_slots"] <= 200
    # keeping every block instead: at call 4 r0 and r2 are cached with no further use; one goes
    keep = P.KVCachePlan(parent, seg, [0, 1, 2, 0, 1], [0, 1, 2, 3, 4], capacity=200, dbc=False)
    assert [e[:2] for e in keep.events(4, 0)] == [("evict", 0), ("refill", 1)]
    assert keep.stats["evictions"] == 2


def test_call_that_cannot_fit_is_rejected():
    with pytest.raises(P.PsattnError) as e:
        P.KVCachePlan([-1, 0], [100, 50], [1], [0], capacity=120)
    assert e.value.name == "PSATTN_E_WORKSPACE"


@pytest.mark.parametrize("name", ["c3", "c4", "c5"])
def test_peak_memory_dynamic_caching_and_adaptive_blocks(name):
    # micro-batches of 8 samples in sample order: releasing blocks at reference count 0 keeps the
    # peak below keeping every block; exact-length blocks below 128-slot pages
    t = W.make(name, tensors=False).tree
    calls = np.arange(len(t.sample_end)) // 8
    big = int(4 * t.num_rows)
    dbc = P.KVCachePlan(t.parent, t.seg_len, t.sample_end, calls, capacity=big)
    keep = P.KVCachePlan(t.parent, t.seg_len, t.sample_end, calls, capacity=big, dbc=False)
    pages = P.KVCachePlan(t.parent, t.seg_len, t.sample_end, calls, capacity=big, block_size=128)
    assert dbc.stats["peak_slots"] < keep.stats["peak_slots"] == t.num_rows
    assert dbc.stats["peak_slots"] < pages.stats["peak_slots"]
    assert np.all(np.diff(keep.used_per_call) >= 0)                               # nothing released early
