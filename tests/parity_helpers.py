"""Shared helpers of the GPU parity tests: run the HIP path, run the oracle, compare."""
import numpy as np

import oracle as O
from paper_2608_25683_amd import workloads as W

TOL = {"bf16": (2e-2, 5e-3), "fp32": (1e-5, 1e-5)}   # (max-abs, relative L2) per output tensor


def run_gpu(wl, opts=None, reps=1):
    """Forward + backward through the C ABI; returns float64 numpy outputs (dK/dV in pool layout)."""
    import torch
    from paper_2608_25683_amd import psattn as P
    tree = P.Tree.from_workload(wl, opts=opts, device="cuda")
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    Q = torch.from_numpy(wl.Q).to("cuda").to(dt)
    K = torch.from_numpy(wl.K_pool).to("cuda").to(dt)
    V = torch.from_numpy(wl.V_pool).to("cuda").to(dt)
    dO = torch.from_numpy(wl.dO).to("cuda").to(dt)
    outs = []
    for _ in range(reps):
        Og, LSEg = P.psattn_fwd(tree, Q, K, V)
        dQ, dK, dV = P.psattn_bwd(tree, Q, K, V, Og, LSEg, dO)
        torch.cuda.synchronize()
        outs.append(tuple(x.float().cpu().numpy().astype(np.float64) for x in (Og, LSEg, dQ, dK, dV)))
    return outs if reps > 1 else outs[0]


def run_oracle(wl):
    """Expanded fp64 oracle; dK/dV mapped to pool slots (pad slots 0)."""
    t = wl.tree
    Of, LSE = O.forward(t.parent, t.seg_len, t.row_off, t.sample_end, wl.Q, wl.K, wl.V, wl.scale)
    dQ, dK, dV = O.backward(t.parent, t.seg_len, t.row_off, t.sample_end, wl.Q, wl.K, wl.V, wl.dO, wl.scale)
    slots = t.row_slots()
    dKp = np.zeros((t.pool_slots,) + dK.shape[1:])
    dVp = np.zeros_like(dKp)
    dKp[slots] = dK
    dVp[slots] = dV
    return Of, LSE, dQ, dKp, dVp


def compare(name, got, ref, dtype, mask=None):
    """max|g-r| <= tau_abs and ||g-r||_2 / ||r||_2 <= tau_rel; returns (maxabs, rel)."""
    tau_abs, tau_rel = TOL[dtype]
    g = got if mask is None else got[mask]
    r = ref if mask is None else ref[mask]
    assert np.all(np.isfinite(g)), f"{name}: non-finite values"
    err = np.abs(g - r)
    maxabs = float(err.max()) if err.size else 0.0
    den = float(np.linalg.norm(r))
    rel = float(np.linalg.norm(g - r) / den) if den > 0 else float(np.linalg.norm(g - r))
    assert maxabs <= tau_abs and rel <= tau_rel, f"{name}: max-abs {maxabs:.3g} (<= {tau_abs}), rel-L2 {rel:.3g} (<= {tau_rel})"
    return maxabs, rel


# softmax rows renormalised with the GPU's LSE sum to 1: sum_j exp(S_ij - LSE_gpu,i) equals
# exp(LSE_i - LSE_gpu,i) with the fp64 LSE_i of the oracle.  fp32: the bound of the fp32 parity
# (an LSE error of 1e-5 moves the sum by 1e-5; an fp32 LSE near 10 is itself only good to 5e-7)
ROWSUM_TOL = {"bf16": 1e-2, "fp32": 1e-5}


def check_rowsums(lse_gpu, lse_ref, dtype):
    dev = np.abs(np.exp(lse_ref - lse_gpu) - 1.0)
    worst = float(dev.max()) if dev.size else 0.0
    assert worst <= ROWSUM_TOL[dtype], f"softmax rows with the GPU LSE sum to 1 +- {worst:.3g} (<= {ROWSUM_TOL[dtype]})"
    return worst


def check_full(wl, gpu, ref):
    Og, LSEg, dQg, dKg, dVg = gpu
    Or, LSEr, dQr, dKr, dVr = ref
    res = {}
    for name, g, r in (("O", Og, Or), ("LSE", LSEg, LSEr), ("dQ", dQg, dQr), ("dK", dKg, dKr), ("dV", dVg, dVr)):
        res[name] = compare(name, g, r, wl.dtype)
    res["rowsum"] = check_rowsums(LSEg, LSEr, wl.dtype)
    # pool slots holding no token get exactly zero
    pad = np.setdiff1d(np.arange(wl.tree.pool_slots), wl.tree.row_slots())
    assert np.all(dKg[pad] == 0) and np.all(dVg[pad] == 0)
    return res


def sample_rows(wl, n_random=24, seed=0):
    """Rows at node starts/ends, tile edges and random positions."""
    t = wl.tree
    rng = np.random.default_rng(seed)
    rows = set()
    for n in range(t.num_nodes):
        r0, L = int(t.row_off[n]), int(t.seg_len[n])
        for a in (0, L - 1, min(L - 1, 31), min(L - 1, 32), min(L - 1, 63), min(L - 1, 64)):
            rows.add(r0 + a)
    rows = sorted(rows)
    if len(rows) > 48:
        rows = sorted(rng.choice(rows, 48, replace=False).tolist())
    rows += rng.integers(0, t.num_rows, n_random).tolist()
    return np.unique(np.asarray(rows, dtype=np.int64))


def sample_keys(wl, seed=0, per_node=3, max_nodes=4):
    """Key rows: first/last/random key of the root(s) and of a few other nodes."""
    t = wl.tree
    rng = np.random.default_rng(seed)
    nodes = [int(n) for n in np.where(t.parent < 0)[0][:2]]
    others = [n for n in range(t.num_nodes) if n not in nodes]
    nodes += [int(x) for x in rng.choice(others, min(len(others), max_nodes - len(nodes)), replace=False)] if others else []
    keys = []
    for n in nodes:
        r0, L = int(t.row_off[n]), int(t.seg_len[n])
        keys += [r0, r0 + L - 1] + [r0 + int(x) for x in rng.integers(0, L, per_node - 2)]
    return np.unique(np.asarray(keys, dtype=np.int64))


def check_sampled(wl, gpu, kv_heads=(0,), seed=0):
    """Full-size parity on sampled outputs evaluated one by one by the oracle."""
    Og, LSEg, dQg, dKg, dVg = gpu
    t = wl.tree
    ti = O.TreeIndex(t.parent, t.seg_len, t.row_off)
    rows = sample_rows(wl, seed=seed)
    heads = list(range(wl.hq))
    o_r, lse_r = O.rows_forward(ti, wl.Q, wl.K, wl.V, wl.scale, rows, heads)
    dq_r = O.rows_dq(ti, wl.Q, wl.K, wl.V, wl.dO, wl.scale, rows, heads)
    res = {"O": compare("O", Og[rows], o_r, wl.dtype), "LSE": compare("LSE", LSEg[:, rows], lse_r, wl.dtype),
           "rowsum": check_rowsums(LSEg[:, rows], lse_r, wl.dtype), "dQ": compare("dQ", dQg[rows], dq_r, wl.dtype)}
    keys = sample_keys(wl, seed=seed)
    slots = t.row_slots()[keys]
    dk_g, dv_g, dk_r, dv_r = [], [], [], []
    for g in kv_heads:
        dk, dv = O.keys_dkdv(ti, wl.Q, wl.K, wl.V, wl.dO, wl.scale, keys, g)
        dk_r.append(dk)
        dv_r.append(dv)
        dk_g.append(dKg[slots, g])
        dv_g.append(dVg[slots, g])
    res["dK"] = compare("dK", np.stack(dk_g), np.stack(dk_r), wl.dtype)
    res["dV"] = compare("dV", np.stack(dv_g), np.stack(dv_r), wl.dtype)
    return res


def check_identities(wl, gpu):
    """Exact identities of the backward, checked at any size (fp64 sums of the GPU outputs)."""
    Og, LSEg, dQg, dKg, dVg = gpu
    t = wl.tree
    G = wl.hq // wl.hkv
    slots = t.row_slots()
    Q, dO = wl.Q.astype(np.float64), wl.dO.astype(np.float64)
    K, V = wl.K.astype(np.float64), wl.V.astype(np.float64)
    dK, dV = dKg[slots], dVg[slots]
    n = len(slots)
    rel = TOL[wl.dtype][1]
    nrm = np.linalg.norm
    # Each bound follows from the relative-L2 parity bound by Cauchy-Schwarz.
    for g in range(wl.hkv):
        hs = slice(g * G, (g + 1) * G)
        # sum_j dK_j = 0
        assert np.max(np.abs(dK[:, g].sum(0))) <= np.sqrt(n) * rel * nrm(dK[:, g])
        # sum_j dV_j = sum_i sum_{h in group} dO_i^h
        assert np.max(np.abs(dV[:, g].sum(0) - dO[:, hs].sum((0, 1)))) <= np.sqrt(n) * rel * nrm(dV[:, g])
        # sum <q, dQ> = sum <k, dK>
        a, b = np.sum(Q[:, hs] * dQg[:, hs]), np.sum(K[:, g] * dK[:, g])
        assert abs(a - b) <= rel * (nrm(Q[:, hs]) * nrm(dQg[:, hs]) + nrm(K[:, g]) * nrm(dK[:, g]))
        # sum <v, dV> = sum <dO, O>
        a, b = np.sum(V[:, g] * dV[:, g]), np.sum(dO[:, hs] * Og[:, hs])
        assert abs(a - b) <= rel * (nrm(V[:, g]) * nrm(dV[:, g]) + nrm(dO[:, hs]) * nrm(Og[:, hs]))
