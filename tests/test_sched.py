"""Host scheduling through the C ABI (Sec. 4.2 workload model and greedy placement, Sec. 4.3
token-wise micro-batching).

* Eq. "single_sequence" T = a1 l_suf l + a2 l_suf + a3: the fit recovers known coefficients
  exactly and is the least-squares solution on noisy data (residual orthogonal to the features).
* Group workloads count each sequence's prefix cached by its group's earlier sequences.
* Greedy placement: a worked example, whole groups, and the longest-processing-time bound
  (makespan <= (4/3 - 1/(3m)) of the optimum, found by brute force on small instances).
* Token-wise micro-batching: the refined forest holds every token once, every refined node is
  computed in exactly one micro-batch, micro-batches stay within the budget (the last takes the
  rest), a sequence is cut exactly when it would overflow, a long sequence splits into chunks of
  near-equal workload, and the result drives the KV cache manager into valid calls.
"""
import itertools

import numpy as np
import pytest

from paper_2608_25683_amd import workloads as W

P = pytest.importorskip("paper_2608_25683_amd.psattn")
ALPHA = np.array([2e-6, 3e-3, 0.5])


def T(a, l_suf, l):
    return a[0] * l_suf * l + a[1] * l_suf + a[2]


def test_fit_recovers_coefficients():
    rng = np.random.default_rng(0)
    l = rng.integers(64, 8192, 40).astype(float)
    l_suf = np.floor(l * rng.uniform(0.05, 1.0, 40))
    t = T(ALPHA, l_suf, l)
    a = P.sched_fit(l_suf, l, t)
    assert np.allclose(a, ALPHA, rtol=1e-7, atol=1e-12)
    noisy = t * (1 + 0.05 * rng.standard_normal(40))
    a = P.sched_fit(l_suf, l, noisy)
    X = np.stack([l_suf * l, l_suf, np.ones_like(l)], 1)
    r = X @ a - noisy
    assert np.all(np.abs(X.T @ r) <= 1e-6 * np.abs(X.T @ noisy))      # normal equations
    with pytest.raises(P.PsattnError):
        P.sched_fit([10, 10, 10], [20, 20, 20], [1, 1, 1])               # degenerate: one point


def test_group_costs_count_cached_prefix():
    # group 0: root(100) -> a(20), root -> b(30); group 1: its own root(50) -> c(10)
    parent, seg = [-1, 0, 0, -1, 3], [100, 20, 30, 50, 10]
    ends, groups = [1, 2, 4], [0, 0, 1]
    c = P.sched_group_costs(parent, seg, ends, groups, 2, ALPHA)
    assert c[0] == pytest.approx(T(ALPHA, 120, 120) + T(ALPHA, 30, 130))   # the root is cached for b
    assert c[1] == pytest.approx(T(ALPHA, 60, 60))


def test_greedy_placement_example_and_bound():
    w, load = P.sched_place([7, 5, 4, 3, 3, 2], 2)
    assert w.tolist() == [0, 1, 1, 0, 1, 0] and load.tolist() == [12, 12]
    rng = np.random.default_rng(1)
    for trial in range(40):
        m = int(rng.integers(2, 4))
        costs = rng.integers(1, 50, int(rng.integers(m + 1, 9))).astype(float)
        w, load = P.sched_place(costs, m)
        assert np.allclose([costs[w == k].sum() for k in range(m)], load)     # every group on one worker
        opt = min(max(sum(costs[i] for i in range(len(costs)) if a[i] == k) for k in range(m))
                  for a in itertools.product(range(m), repeat=len(costs)))
        assert load.max() <= (4 / 3 - 1 / (3 * m)) * opt + 1e-9


def _check_microbatch(parent, seg, ends, M, alpha=ALPHA):
    mb = P.sched_microbatch(parent, seg, ends, alpha, M)
    parent, seg = np.asarray(parent), np.asarray(seg)
    # the refined nodes tile every original node exactly
    for n in range(len(seg)):
        pieces = sorted((o, L) for o, L, s in zip(mb["src_offset"], mb["seg_len"], mb["src_node"]) if s == n)
        assert pieces[0][0] == 0 and all(a[0] + a[1] == b[0] for a, b in zip(pieces, pieces[1:]))
        assert pieces[-1][0] + pieces[-1][1] == seg[n]
    rp = mb["parent"]
    path = lambda e: (path(rp[e]) if rp[e] >= 0 else []) + [int(e)]
    # every refined node is computed in exactly one micro-batch: the first chunk that reaches it
    first = {}
    for e, k in zip(mb["chunk_end"], mb["chunk_micro_batch"]):
        for r in path(e):
            first.setdefault(r, k)
    assert set(first) == set(range(len(rp)))
    # each original sample's chunks: consecutive micro-batches, the last chunk ends at the sample's end
    for s, e in enumerate(ends):
        ks = [k for k, cs in zip(mb["chunk_micro_batch"], mb["chunk_sample"]) if cs == s]
        assert ks == sorted(ks)
        last = [c for c, cs in zip(mb["chunk_end"], mb["chunk_sample"]) if cs == s][-1]
        assert mb["src_node"][last] == e and mb["src_offset"][last] + mb["seg_len"][last] == seg[e]
    # budgets: total workload / M, the last micro-batch takes the rest
    done, total = set(), 0.0
    for e in ends:
        p = []
        x = e
        while x >= 0:
            p.append(x)
            x = parent[x]
        l = sum(seg[q] for q in p)
        h = sum(seg[q] for q in p if q in done)
        done |= set(p)
        total += T(alpha, l - h, l)
    costs = mb["micro_batch_cost"]
    assert np.all(costs[:-1] <= total / M * (1 + 1e-9))
    return mb, total


def test_long_sequence_splits_into_equal_work_chunks():
    # the budget is a quarter of the whole sequence's Eq. 1 workload; chunks see shorter key ranges
    # than the whole sequence, so three chunks fill the first three micro-batches and the last one
    # gets no work
    mb, total = _check_microbatch([-1], [10000], [0], 4)
    assert len(mb["chunk_end"]) == 3 and mb["chunk_micro_batch"].tolist() == [0, 1, 2]
    c = mb["micro_batch_cost"]
    assert np.all(np.abs(c[:-1] - total / 4) <= ALPHA[0] * 10000 * 2 + ALPHA[1])   # full up to one token
    lens = mb["seg_len"]
    assert np.all(np.diff(lens) < 0)            # later chunks see longer prefixes: fewer tokens each


def test_sequence_cut_exactly_when_it_would_overflow():
    # two sequences: the first fills about 70% of one of two micro-batches' budget, the second is cut
    parent, seg, ends = [-1, -1], [2000, 3000], [0, 1]
    mb, total = _check_microbatch(parent, seg, ends, 2)
    assert mb["chunk_sample"].tolist() == [0, 1, 1] and mb["chunk_micro_batch"].tolist() == [0, 0, 1]
    # the cut is where a1 x (x) + a2 x + a3 first exceeds what the first sequence left
    left = total / 2 - T(ALPHA, 2000, 2000)
    x = int(mb["seg_len"][1])
    assert T(ALPHA, x, x) <= left < T(ALPHA, x + 1, x + 1)


@pytest.mark.parametrize("name,M", [("c3", 6), ("c4", 8), ("c5", 10)])
def test_microbatches_drive_the_cache_manager(name, M):
    t = W.make(name, tensors=False).tree
    mb, _ = _check_microbatch(t.parent, t.seg_len, t.sample_end, M)
    plan = P.KVCachePlan(mb["parent"], mb["seg_len"], mb["chunk_end"], mb["chunk_micro_batch"],
                         capacity=int(t.num_rows))
    assert plan.num_calls == len(mb["micro_batch_cost"])
    computed = set()
    for c in range(plan.num_calls):
        x = plan.call(c)
        tree = P.Tree(parent=x["parent"], seg_len=x["seg_len"], row_off=x["row_off"], blk_ptr=x["blk_ptr"],
                      blk_base=x["blk_base"], blk_cap=x["blk_cap"], blk_len=x["blk_len"], blk_pos=x["blk_pos"],
                      pool_slots=x["pool_slots"], sample_end=x["sample_end"], hq=8, hkv=2, head_dim=128,
                      softmax_scale=0.088)
        internal = {int(n) for n, r in zip(x["node_ids"], x["row_off"]) if r >= 0}
        assert not internal & computed
        computed |= internal
        assert tree.num_rows == sum(int(mb["seg_len"][n]) for n in internal)
    assert computed == set(range(len(mb["parent"])))
