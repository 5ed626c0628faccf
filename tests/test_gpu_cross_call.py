"""Cross-call prefix reuse on the GPU (Sec. 4.1.1 inter-batch sharing, Sec. 4.1.2 self-sequence
sharing, Sec. 5.2 reference counts): a forest processed over several calls, each later call
reading the cached K/V of nodes an earlier call computed and adding its share of their dK/dV to
the same fp32 accumulators.  After the last call the outputs of every call and the accumulated
dK/dV match the fp64 oracle on the whole forest, at the bf16 tolerances.
"""
import sys

import numpy as np
import pytest

from paper_2608_25683_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

import parity_helpers as H  # noqa: E402


def _run_calls(forest, calls, opts=None):
    """Run the calls in order on one pool with shared dK/dV; return forest-shaped outputs."""
    from paper_2608_25683_amd import psattn as P
    dev = torch.device("cuda")
    t = forest.tree
    K = torch.from_numpy(forest.K_pool).to(dev).to(torch.bfloat16)
    V = torch.from_numpy(forest.V_pool).to(dev).to(torch.bfloat16)
    dK = torch.full((t.pool_slots, forest.hkv, forest.d), float("nan"), dtype=torch.float32, device=dev)
    dV = torch.full_like(dK, float("nan"))
    Of = np.zeros((t.num_rows, forest.hq, forest.d))
    LSEf = np.zeros((forest.hq, t.num_rows))
    dQf = np.zeros((t.num_rows, forest.hq, forest.d))
    for ends, external in calls:
        call, rows = W.call_subset(forest, ends, external)
        tree = P.Tree.from_workload(call, opts=opts, device="cuda")
        Q = torch.from_numpy(call.Q).to(dev).to(torch.bfloat16)
        dO = torch.from_numpy(call.dO).to(dev).to(torch.bfloat16)
        O, LSE = P.psattn_fwd(tree, Q, K, V)
        dQ, _, _ = P.psattn_bwd(tree, Q, K, V, O, LSE, dO, dK=dK, dV=dV)
        torch.cuda.synchronize()
        Of[rows] = O.float().cpu().numpy()
        LSEf[:, rows] = LSE.cpu().numpy()
        dQf[rows] = dQ.cpu().numpy()
    return Of, LSEf, dQf, dK.cpu().numpy().astype(np.float64), dV.cpu().numpy().astype(np.float64)


def _compare(forest, got, ref):
    t = forest.tree
    slots = t.row_slots()
    res = {}
    for i, name in enumerate(("O", "LSE", "dQ")):
        res[name] = H.compare(name, got[i], ref[i], "bf16")
    for i, name in ((3, "dK"), (4, "dV")):
        res[name] = H.compare(name, got[i][slots], ref[i][slots], "bf16")
    return res


FOREST = dict(parent=[-1, 0, 0, 1, 0, 1], seg=[300, 150, 70, 90, 20, 33], samples=[3, 2, 4, 5])


@pytest.mark.parametrize("opts", [None, {"fwd_kv_split": 128, "bwd_q_chunk": 32}])
def test_inter_batch_sharing(opts):
    # call 1: the first sample's path (root, node 1, node 3); call 2: the other samples, with the
    # nodes of call 1 cached
    f = FOREST
    forest = W.custom(f["parent"], f["seg"], f["samples"], hq=8, hkv=2, d=128, dtype="bf16", seed=31,
                      block_policy=lambda L: W.blocks_fixed(L, 64))
    t = forest.tree
    first = [int(t.sample_end[0])]
    done = set(m for e in first for m in t.path(e))
    rest = [int(t.sample_end[s]) for s in range(1, len(t.sample_end))]
    print(f"inter-batch: call 1 ends {first}, call 2 ends {rest} with {sorted(done)} cached", file=sys.stderr)
    got = _run_calls(forest, [(first, []), (rest, sorted(done))], opts=opts)
    res = _compare(forest, got, H.run_oracle(forest))
    print(f"inter-batch {res}", file=sys.stderr)


def test_three_micro_batches():
    # one sample per call, each later call caching everything computed before it
    f = FOREST
    forest = W.custom(f["parent"], f["seg"], f["samples"], hq=10, hkv=2, d=128, dtype="bf16", seed=32,
                      block_policy=W.blocks_exact)
    t = forest.tree
    calls, done = [], set()
    for s in range(len(t.sample_end)):
        e = int(t.sample_end[s])
        calls.append(([e], sorted(done & set(t.path(e)))))
        done |= set(t.path(e))
    got = _run_calls(forest, calls)
    res = _compare(forest, got, H.run_oracle(forest))
    print(f"micro-batches {res}", file=sys.stderr)


def test_self_sequence_sharing():
    # one 900-token sequence as four chunks (a chain), one call per chunk: chunk c attends to the
    # cached chunks 0..c-1 and adds to their dK/dV
    forest = W.custom([-1, 0, 1, 2], [260, 230, 150, 260], [3], hq=8, hkv=2, d=64, dtype="bf16", seed=33,
                      block_policy=W.blocks_greedy)
    calls = [([c], list(range(c))) for c in range(4)]
    got = _run_calls(forest, calls, opts={"bwd_q_chunk": 64})
    res = _compare(forest, got, H.run_oracle(forest))
    print(f"chunked {res}", file=sys.stderr)


def _run_managed(forest, parent, seg_len, ends, calls, node_rows, capacity):
    """Calls planned by the KV cache manager over a (possibly refined) forest whose node r holds the
    forest rows node_rows(r); the test plays the caller: it writes K/V into new blocks, zeroes the
    dK/dV of refilled ones, and flushes dK/dV of evicted and freed blocks into per-row sums."""
    from paper_2608_25683_amd import psattn as P
    plan = P.KVCachePlan(parent, seg_len, ends, calls, capacity=capacity)
    t = forest.tree
    dev = torch.device("cuda")
    hkv, d = forest.hkv, forest.d
    Kp = torch.zeros((capacity, hkv, d), dtype=torch.bfloat16, device=dev)
    Vp = torch.zeros_like(Kp)
    dK = torch.zeros((capacity, hkv, d), dtype=torch.float32, device=dev)
    dV = torch.zeros_like(dK)
    Kt = torch.from_numpy(forest.K).to(dev).to(torch.bfloat16)     # node-packed (forest rows)
    Vt = torch.from_numpy(forest.V).to(dev).to(torch.bfloat16)
    slots_of = {}
    gK = np.zeros((t.num_rows, hkv, d))
    gV = np.zeros((t.num_rows, hkv, d))
    Of = np.zeros((t.num_rows, forest.hq, d))
    LSEf = np.zeros((forest.hq, t.num_rows))
    dQf = np.zeros((t.num_rows, forest.hq, d))

    def flush(n):
        s_ = torch.from_numpy(slots_of[n]).to(dev)
        gK[node_rows(n)] += dK[s_].cpu().numpy()
        gV[node_rows(n)] += dV[s_].cpu().numpy()

    for c in range(plan.num_calls):
        x = plan.call(c)
        ev = {e[1]: e[0] for e in plan.events(c, 0)}
        for kind, n, _, _, _ in plan.events(c, 0):
            if kind == "evict":
                flush(n)
        for i, n in enumerate(x["node_ids"]):
            new = np.concatenate([np.arange(x["blk_base"][b], x["blk_base"][b] + x["blk_len"][b])
                                  for b in range(x["blk_ptr"][i], x["blk_ptr"][i + 1])])
            if ev.get(int(n)) in ("alloc", "refill"):
                s_ = torch.from_numpy(new).to(dev)
                r = torch.from_numpy(node_rows(int(n))).to(dev)
                Kp[s_] = Kt[r]
                Vp[s_] = Vt[r]
                if ev[int(n)] == "refill":
                    dK[s_] = 0
                    dV[s_] = 0
            slots_of[int(n)] = new
        tree = P.Tree(parent=x["parent"], seg_len=x["seg_len"], row_off=x["row_off"], blk_ptr=x["blk_ptr"],
                      blk_base=x["blk_base"], blk_cap=x["blk_cap"], blk_len=x["blk_len"], blk_pos=x["blk_pos"],
                      pool_slots=x["pool_slots"], sample_end=x["sample_end"], hq=forest.hq, hkv=hkv, head_dim=d,
                      softmax_scale=forest.scale, device="cuda")
        frows = np.concatenate([node_rows(int(n)) for i, n in enumerate(x["node_ids"]) if x["row_off"][i] >= 0])
        Q = torch.from_numpy(forest.Q[frows]).to(dev).to(torch.bfloat16)
        dO = torch.from_numpy(forest.dO[frows]).to(dev).to(torch.bfloat16)
        Og, LSEg = P.psattn_fwd(tree, Q, Kp, Vp)
        dQ, _, _ = P.psattn_bwd(tree, Q, Kp, Vp, Og, LSEg, dO, dK=dK, dV=dV)
        torch.cuda.synchronize()
        Of[frows] = Og.float().cpu().numpy()
        LSEf[:, frows] = LSEg.cpu().numpy()
        dQf[frows] = dQ.cpu().numpy()
        for kind, n, _, _, _ in plan.events(c, 1):
            if kind == "free":
                flush(n)
    return plan, (Of, LSEf, dQf, gK, gV)


def _oracle_rows(forest):
    import oracle as O
    t = forest.tree
    Or, LSEr = O.forward(t.parent, t.seg_len, t.row_off, t.sample_end, forest.Q, forest.K, forest.V, forest.scale)
    dQr, dKr, dVr = O.backward(t.parent, t.seg_len, t.row_off, t.sample_end, forest.Q, forest.K, forest.V, forest.dO,
                               forest.scale)
    return Or, LSEr, dQr, dKr, dVr


def _compare_rows(got, ref):
    return {name: H.compare(name, g, r, "bf16") for name, g, r in zip(("O", "LSE", "dQ", "dK", "dV"), got, ref)}


def test_kv_cache_manager_schedule_with_eviction():
    # the adaptive KV cache manager drives the calls: one sample per call, a pool too small to keep
    # every shared block, so a block is evicted (its partial dK/dV flushed) and refilled later
    # (K/V written again, dK/dV restarted at zero); the flushed gradients of every node add up to
    # the whole forest's dK/dV
    forest = W.custom([-1, 0, 0, -1, 3, 3, 1], [200, 60, 90, 180, 40, 70, 50], [6, 2, 4, 5], hq=8, hkv=2, d=128,
                      dtype="bf16", seed=41, block_policy=W.blocks_exact)
    t = forest.tree
    # calls: tree A (root 0) | tree B (root 3) | tree A again | tree B again; at call 2 only B's
    # root can make room, although call 3 reads it
    rows = lambda n: np.arange(int(t.row_off[n]), int(t.row_off[n] + t.seg_len[n]))
    plan, got = _run_managed(forest, t.parent, t.seg_len, t.sample_end, [0, 2, 1, 3], rows, 420)
    assert plan.stats["evictions"] >= 1 and plan.stats["refilled_tokens"] > 0
    res = _compare_rows(got, _oracle_rows(forest))
    print(f"kv-cache schedule {plan.stats} {res}", file=sys.stderr)


def test_token_wise_micro_batches():
    # Sec. 4.3: the forest's samples cut into 5 micro-batches of near-equal Eq. 1 workload, long
    # sequences split at token boundaries (the refined forest's nodes are pieces of the forest's);
    # the KV cache manager plans the calls and the op runs them
    from paper_2608_25683_amd import psattn as P
    forest = W.custom([-1, 0, 0, 1, -1, 4], [700, 300, 120, 900, 250, 60], [3, 2, 5], hq=8, hkv=2, d=128,
                      dtype="bf16", seed=43, block_policy=W.blocks_exact)
    t = forest.tree
    mb = P.sched_microbatch(t.parent, t.seg_len, t.sample_end, [2e-6, 3e-3, 0.5], 5)
    assert len(mb["parent"]) > t.num_nodes      # some sequence was cut inside a node
    rows = lambda r: np.arange(int(t.row_off[mb["src_node"][r]] + mb["src_offset"][r]),
                               int(t.row_off[mb["src_node"][r]] + mb["src_offset"][r] + mb["seg_len"][r]))
    plan, got = _run_managed(forest, mb["parent"], mb["seg_len"], mb["chunk_end"], mb["chunk_micro_batch"], rows,
                             int(t.num_rows))
    res = _compare_rows(got, _oracle_rows(forest))
    print(f"micro-batches {len(mb['micro_batch_cost'])} calls, {len(mb['parent'])} refined nodes: {res}",
          file=sys.stderr)
