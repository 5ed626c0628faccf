"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: central
finite differences, closed forms, torch's scaled_dot_product_attention in
fp64 (with autograd summing duplicated prefix gradients), exact gradient
identities, invariance to how a shared adjoint is split among copies, and
the paper's shared == unshared contract (Sec. 2.5).
"""
import math

import numpy as np
import pytest

import oracle as O
from paper_2608_25683_amd import workloads as W


def tiny_tree(seed, d=4, hq=2, hkv=1):
    """<= 3 nodes, <= 8 tokens each, 2-3 samples sharing a prefix."""
    rng = np.random.default_rng(1000 + seed)
    shapes = [([-1, 0, 0], [1, 2]), ([-1, 0, 1], [1, 2]), ([-1, 0, 0], [0, 1, 2])]
    parent, samples = shapes[seed % 3]
    seg = [int(rng.integers(1, 9)) for _ in parent]
    return W.custom(parent, seg, samples, hq=hq, hkv=hkv, d=d, dtype="fp32", seed=seed, sigma=1.0,
                    block_policy=W.blocks_exact)


def run_oracle(wl, split="owner"):
    t = wl.tree
    Q, K, V, dO = (x.astype(np.float64) for x in (wl.Q, wl.K, wl.V, wl.dO))
    Of, LSE = O.forward(t.parent, t.seg_len, t.row_off, t.sample_end, Q, K, V, wl.scale)
    dQ, dK, dV = O.backward(t.parent, t.seg_len, t.row_off, t.sample_end, Q, K, V, dO, wl.scale, split=split)
    return Of, LSE, dQ, dK, dV


# --------------------------------------------------------------------------- Pi1: finite differences

@pytest.mark.parametrize("seed", range(6))
def test_pi1_finite_differences(seed):
    wl = tiny_tree(seed)
    t = wl.tree
    Q, K, V, dO = (x.astype(np.float64) for x in (wl.Q, wl.K, wl.V, wl.dO))

    def loss(Q_, K_, V_):
        Of, _ = O.forward(t.parent, t.seg_len, t.row_off, t.sample_end, Q_, K_, V_, wl.scale, check_copies=False)
        return float(np.sum(dO * Of))

    _, _, dQ, dK, dV = run_oracle(wl)
    for X, G in ((Q, dQ), (K, dK), (V, dV)):
        fd = np.zeros_like(X)
        for idx in np.ndindex(*X.shape):
            h = 1e-6 * max(1.0, abs(X[idx]))
            xp = X.copy(); xp[idx] += h
            xm = X.copy(); xm[idx] -= h
            args_p = [Q, K, V]; args_m = [Q, K, V]
            which = [Q is X, K is X, V is X].index(True)
            args_p[which] = xp; args_m[which] = xm
            fd[idx] = (loss(*args_p) - loss(*args_m)) / (2 * h)
        err = np.max(np.abs(fd - G)) / max(1e-12, np.max(np.abs(G)))
        assert err <= 1e-6, err


# --------------------------------------------------------------------------- Pi2, Pi3: softmax rows, shared == unshared

@pytest.mark.parametrize("seed", range(8))
def test_pi2_softmax_rows_sum_to_one(seed):
    wl = W.random_forest(seed, max_nodes=8, max_seg=24, d=16, dtype="fp32", sigma=1.0)
    t = wl.tree
    ti = O.TreeIndex(t.parent, t.seg_len, t.row_off)
    _, LSE = O.forward(t.parent, t.seg_len, t.row_off, t.sample_end, wl.Q, wl.K, wl.V, wl.scale)
    G = wl.hq // wl.hkv
    for r in range(t.num_rows):
        n = int(ti.row_node[r])
        keys = ti.path_rows(n)[: int(ti.off[n] + r - ti.row_off[n]) + 1]
        for h in range(wl.hq):
            s = wl.scale * (wl.K[keys, h // G].astype(np.float64) @ wl.Q[r, h].astype(np.float64))
            assert abs(np.exp(s - LSE[h, r]).sum() - 1.0) <= 1e-12


@pytest.mark.parametrize("seed", range(8))
def test_pi3_shared_equals_unshared(seed):
    # forward() raises when two copies of a shared token disagree beyond 1e-12
    wl = W.random_forest(seed, max_nodes=10, max_seg=30, d=16, dtype="fp32", sigma=1.0)
    t = wl.tree
    O.forward(t.parent, t.seg_len, t.row_off, t.sample_end, wl.Q, wl.K, wl.V, wl.scale, tol=1e-12)


def test_pi3_detects_a_broken_mask():
    # the check is live: a wrong (non-causal) mask makes copies disagree
    wl = W.custom([-1, 0, 0], [5, 3, 4], [1, 2], hq=2, hkv=1, d=8, dtype="fp32", seed=3, sigma=1.0)
    t = wl.tree
    orig = O.causal_fwd

    def leaky(q, k, v, scale):
        s = scale * (q @ k.T)
        m = s.max(axis=1, keepdims=True)
        e = np.exp(s - m)
        return (e / e.sum(1, keepdims=True)) @ v, (m + np.log(e.sum(1, keepdims=True)))[:, 0]
    try:
        O.psattn_oracle.causal_fwd = leaky
        with pytest.raises(AssertionError):
            O.psattn_oracle.forward(t.parent, t.seg_len, t.row_off, t.sample_end, wl.Q, wl.K, wl.V, wl.scale)
    finally:
        O.psattn_oracle.causal_fwd = orig


# --------------------------------------------------------------------------- Pi4: torch SDPA special cases

torch = pytest.importorskip("torch")


def _walk_samples(t):
    """Each sample's packed rows in sequence order, and each row's owner sample, found by walking
    parent[] up from the sample's endpoint (independent of the oracle's own expansion)."""
    seqs = []
    row_owner = np.full(t.num_rows, -1, dtype=np.int64)
    for s, e in enumerate(t.sample_end):
        nodes = []
        n = int(e)
        while n != -1:
            nodes.append(n)
            n = int(t.parent[n])
        rows = []
        for n in reversed(nodes):                                      # root first
            rows.extend(range(int(t.row_off[n]), int(t.row_off[n]) + int(t.seg_len[n])))
        rows = np.asarray(rows, dtype=np.int64)
        unowned = rows[row_owner[rows] < 0]
        row_owner[unowned] = s
        seqs.append(rows)
    return seqs, row_owner


def _sdpa_tree(wl, split="owner"):
    """Per-sample SDPA in fp64 through an index-gather; autograd sums duplicate gradients."""
    import torch.nn.functional as F
    t = wl.tree
    G = wl.hq // wl.hkv
    Q = torch.tensor(wl.Q, dtype=torch.float64, requires_grad=True)
    K = torch.tensor(wl.K, dtype=torch.float64, requires_grad=True)
    V = torch.tensor(wl.V, dtype=torch.float64, requires_grad=True)
    dO = torch.tensor(wl.dO, dtype=torch.float64)
    seqs, row_owner = _walk_samples(t)
    loss = 0.0
    outs = []
    for s, rows in enumerate(seqs):
        ri = torch.tensor(rows)
        q = Q[ri].permute(1, 0, 2)                                     # [Hq, L, d]
        k = K[ri].permute(1, 0, 2).repeat_interleave(G, dim=0)         # head h reads kv head h // G
        v = V[ri].permute(1, 0, 2).repeat_interleave(G, dim=0)
        o = F.scaled_dot_product_attention(q, k, v, is_causal=True, scale=wl.scale)
        w = torch.tensor((row_owner[rows] == s).astype(np.float64))
        loss = loss + (o * (dO[ri].permute(1, 0, 2) * w[None, :, None])).sum()
        outs.append((rows, o.detach().permute(1, 0, 2).numpy()))
    loss.backward()
    return outs, Q.grad.numpy(), K.grad.numpy(), V.grad.numpy()


@pytest.mark.parametrize("shape", ["single", "chain", "branch", "gqa_branch"])
def test_pi4_matches_torch_sdpa(shape):
    if shape == "single":
        wl = W.custom([-1], [37], [0], hq=2, hkv=2, d=16, dtype="fp32", seed=1, sigma=1.0)
    elif shape == "chain":
        wl = W.custom([-1, 0, 1], [9, 5, 11], [2], hq=2, hkv=1, d=16, dtype="fp32", seed=2, sigma=1.0)
    elif shape == "branch":
        wl = W.custom([-1, 0, 0, 1], [13, 4, 7, 6], [3, 2, 0], hq=2, hkv=2, d=16, dtype="fp32", seed=3, sigma=1.0)
    else:
        wl = W.custom([-1, 0, 0, 0, 2], [21, 3, 8, 5, 9], [1, 4, 3], hq=6, hkv=2, d=8, dtype="fp32", seed=4, sigma=1.0)
    Of, LSE, dQ, dK, dV = run_oracle(wl)
    outs, gQ, gK, gV = _sdpa_tree(wl)
    for rows, o in outs:
        assert np.max(np.abs(Of[rows] - o)) <= 1e-10
    for a, b in ((dQ, gQ), (dK, gK), (dV, gV)):
        assert np.max(np.abs(a - b)) <= 1e-10


def test_pi4_catches_a_path_order_bug():
    # planted in the oracle: root-to-node paths listed child first; the SDPA pin, which walks
    # parent[] itself, must then disagree
    wl = W.custom([-1, 0, 1], [9, 5, 11], [2, 1], hq=2, hkv=1, d=16, dtype="fp32", seed=2, sigma=1.0)
    orig = O.psattn_oracle.node_paths

    def reversed_paths(parent):
        return [p[::-1] for p in orig(parent)]
    t = wl.tree
    try:
        O.psattn_oracle.node_paths = reversed_paths
        Of, _ = O.forward(t.parent, t.seg_len, t.row_off, t.sample_end, wl.Q.astype(np.float64),
                          wl.K.astype(np.float64), wl.V.astype(np.float64), wl.scale, check_copies=False)
    finally:
        O.psattn_oracle.node_paths = orig
    outs, gQ, gK, gV = _sdpa_tree(wl)
    worst = max(float(np.max(np.abs(Of[rows] - o))) for rows, o in outs)
    assert worst > 1e-3


# --------------------------------------------------------------------------- Pi5: closed forms

def test_pi5_zero_queries_give_uniform_attention():
    wl = W.random_forest(11, max_nodes=9, max_seg=20, d=8, dtype="fp32", sigma=1.0)
    t = wl.tree
    ti = O.TreeIndex(t.parent, t.seg_len, t.row_off)
    Q0 = np.zeros_like(wl.Q)
    Of, LSE = O.forward(t.parent, t.seg_len, t.row_off, t.sample_end, Q0, wl.K, wl.V, wl.scale)
    G = wl.hq // wl.hkv
    for r in range(t.num_rows):
        n = int(ti.row_node[r])
        nvis = int(ti.off[n] + r - ti.row_off[n]) + 1
        keys = ti.path_rows(n)[:nvis]
        for h in range(wl.hq):
            assert abs(LSE[h, r] - math.log(nvis)) <= 1e-12
            assert np.max(np.abs(Of[r, h] - wl.V[keys, h // G].astype(np.float64).mean(0))) <= 1e-12


def test_pi5_constant_values():
    wl = W.random_forest(12, max_nodes=9, max_seg=20, d=8, dtype="fp32", sigma=1.0)
    t = wl.tree
    V = np.broadcast_to(np.linspace(-1, 1, wl.d), wl.V.shape).copy()
    Of, _ = O.forward(t.parent, t.seg_len, t.row_off, t.sample_end, wl.Q, wl.K, V, wl.scale)
    dQ, dK, dV = O.backward(t.parent, t.seg_len, t.row_off, t.sample_end, wl.Q, wl.K, V, wl.dO, wl.scale)
    assert np.max(np.abs(Of - V[0, 0][None, None, :])) <= 1e-12
    assert np.max(np.abs(dQ)) <= 1e-12 and np.max(np.abs(dK)) <= 1e-12


def test_pi5_first_token_of_a_root():
    wl = W.random_forest(13, max_nodes=9, max_seg=20, d=8, dtype="fp32", sigma=1.0)
    t = wl.tree
    Of, LSE = O.forward(t.parent, t.seg_len, t.row_off, t.sample_end, wl.Q, wl.K, wl.V, wl.scale)
    G = wl.hq // wl.hkv
    for n in range(t.num_nodes):
        if t.parent[n] >= 0:
            continue
        r = int(t.row_off[n])
        for h in range(wl.hq):
            assert np.max(np.abs(Of[r, h] - wl.V[r, h // G])) <= 1e-12
            ref = wl.scale * float(wl.Q[r, h].astype(np.float64) @ wl.K[r, h // G].astype(np.float64))
            assert abs(LSE[h, r] - ref) <= 1e-12


# --------------------------------------------------------------------------- Pi6, Pi7: identities, split invariance

@pytest.mark.parametrize("seed", range(4))
def test_pi6_gradient_identities(seed):
    wl = W.random_forest(20 + seed, max_nodes=10, max_seg=30, hq=6, hkv=2, d=16, dtype="fp32", sigma=1.0)
    Of, _, dQ, dK, dV = run_oracle(wl)
    G = wl.hq // wl.hkv
    Q, K, V, dO = (x.astype(np.float64) for x in (wl.Q, wl.K, wl.V, wl.dO))
    for g in range(wl.hkv):
        hs = slice(g * G, (g + 1) * G)
        assert np.max(np.abs(dK[:, g].sum(0))) <= 1e-12
        assert np.max(np.abs(dV[:, g].sum(0) - dO[:, hs].sum((0, 1)))) <= 1e-11
        assert abs(np.sum(Q[:, hs] * dQ[:, hs]) - np.sum(K[:, g] * dK[:, g])) <= 1e-11
        assert abs(np.sum(V[:, g] * dV[:, g]) - np.sum(dO[:, hs] * Of[:, hs])) <= 1e-11


@pytest.mark.parametrize("seed", range(4))
def test_pi7_adjoint_split_invariance(seed):
    wl = W.random_forest(30 + seed, max_nodes=10, max_seg=25, d=16, dtype="fp32", sigma=1.0)
    a = run_oracle(wl, "owner")[2:]
    b = run_oracle(wl, "uniform")[2:]
    for x, y in zip(a, b):
        assert np.max(np.abs(x - y)) <= 1e-12


# --------------------------------------------------------------------------- point evaluators == expanded oracle

@pytest.mark.parametrize("seed", range(5))
def test_point_evaluators_match_expanded_oracle(seed):
    wl = W.random_forest(40 + seed, max_nodes=10, max_seg=30, hq=4, hkv=2, d=16, dtype="fp32", sigma=1.0,
                         shuffle_rows=(seed % 2 == 1))
    t = wl.tree
    Of, LSE, dQ, dK, dV = run_oracle(wl)
    ti = O.TreeIndex(t.parent, t.seg_len, t.row_off)
    rows = np.arange(t.num_rows)
    heads = list(range(wl.hq))
    o2, l2 = O.rows_forward(ti, wl.Q, wl.K, wl.V, wl.scale, rows, heads)
    assert np.max(np.abs(o2 - Of)) <= 1e-12 and np.max(np.abs(l2 - LSE)) <= 1e-12
    dq2 = O.rows_dq(ti, wl.Q, wl.K, wl.V, wl.dO, wl.scale, rows, heads)
    assert np.max(np.abs(dq2 - dQ)) <= 1e-12
    for g in range(wl.hkv):
        dk2, dv2 = O.keys_dkdv(ti, wl.Q, wl.K, wl.V, wl.dO, wl.scale, rows, g)
        assert np.max(np.abs(dk2 - dK[:, g])) <= 1e-12
        assert np.max(np.abs(dv2 - dV[:, g])) <= 1e-12
