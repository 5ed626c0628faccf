"""Shared helpers of the GPU parity tests: run the HIP path, run the oracle, compare."""
import os

import numpy as np

import oracle as O
from paper_2608_25683_amd import workloads as W

TOL = {"bf16": (2e-2, 5e-3), "fp32": (1e-5, 1e-5)}   # (max-abs, relative L2) per output tensor


def run_gpu(wl, opts=None, reps=1, residual=True):
    """Forward + backward through the C ABI; returns float64 numpy outputs (dK/dV in pool layout).
    bf16: with residual, the forward's rounding residual of O goes to the backward (O_lo)."""
    import torch
    from paper_2608_25683_amd import psattn as P
    tree = P.Tree.from_workload(wl, opts=opts, device="cuda")
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    Q = torch.from_numpy(wl.Q).to("cuda").to(dt)
    K = torch.from_numpy(wl.K_pool).to("cuda").to(dt)
    V = torch.from_numpy(wl.V_pool).to("cuda").to(dt)
    dO = torch.from_numpy(wl.dO).to("cuda").to(dt)
    O_lo = torch.empty_like(Q) if (residual and wl.dtype == "bf16") else None
    outs = []
    for _ in range(reps):
        Og, LSEg = P.psattn_fwd(tree, Q, K, V, O_lo=O_lo)
        dQ, dK, dV = P.psattn_bwd(tree, Q, K, V, Og, LSEg, dO, O_lo=O_lo)
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


# --------------------------------------------------------------------------- full-size parity, element by element
#
# On a full-size workload the oracle evaluates, for every kv head: every key of the first and the
# last 128-key tile of the most-shared node (the one whose subtree holds the most rows: the c2
# root is read by every row), the first and the last tile of one leaf, and -- from the same
# per-row forward -- O and LSE of every row that consumes the most-shared node, for every query
# head.  dQ is checked on every row of the first and the last query tile of the most-shared node
# and of the leaf.  Two complete slices are evaluated besides and gated on their own: dK and dV
# of every key of the most-shared node and of the leaf on kv head 0 (the c2 root's 4096 keys,
# each summed over all its consumers; on c4 and c2-small through partial tiles and the chunk
# sum), and dQ of every row of one branch (a leaf of at most 1024 rows) for the query heads of kv
# head 0.  The kv heads run in parallel worker processes (numpy only; the inputs and the GPU
# outputs are shared through memory-mapped files).

def _most_shared_and_leaf(t):
    ti = O.TreeIndex(t.parent, t.seg_len, t.row_off)
    sub_rows = [sum(int(t.seg_len[c]) for c in ti.subtree(n)) for n in range(t.num_nodes)]
    shared = int(np.argmax(sub_rows))
    leaves = [n for n in ti.subtree(shared) if not ti.children[n] and n != shared]
    leaf = max(leaves, key=lambda n: (int(t.seg_len[n]), n)) if leaves else shared
    return ti, shared, leaf


def _tiles(r0, L, w):
    """Rows of the first and the last w-row tile of a node of L rows starting at row r0."""
    first = list(range(r0, r0 + min(w, L)))
    last = list(range(r0 + (L - 1) // w * w, r0 + L))
    return sorted(set(first) | set(last))


def _stats(g, r):
    e = np.abs(g - r)
    return (float(e.max()) if e.size else 0.0, float(np.sum((g - r) ** 2)), float(np.sum(r ** 2)))


def _full_size_worker(job):
    """One kv head: oracle values of the selected outputs, compared with the GPU's (partial stats)."""
    from threadpoolctl import threadpool_limits
    with threadpool_limits(limits=job["threads"]):
        return _full_size_job(job)


def _full_size_job(job):
    import numpy as _np
    d = {k: _np.load(v, mmap_mode="r") for k, v in job["files"].items()}
    ti = O.TreeIndex(d["parent"], d["seg_len"], d["row_off"])
    g, G, scale = job["g"], job["G"], job["scale"]
    heads = list(range(g * G, (g + 1) * G))
    fo = {}
    dk, dv = O.keys_dkdv(ti, d["Q"], d["K"], d["V"], d["dO"], scale, job["keys"], g, forward_out=fo)
    slots = d["row_slots"][job["keys"]]
    out = {"dK": _stats(_np.asarray(d["gdK"][slots, g], _np.float64), dk),
           "dV": _stats(_np.asarray(d["gdV"][slots, g], _np.float64), dv)}
    if job["complete"]:   # job["keys"] is then the complete slice
        out["dK complete"], out["dV complete"] = out["dK"], out["dV"]
    o_st, l_st, rs = [], [], 0.0
    for m, (cons, Oc, LSEc) in fo.items():
        o_st.append(_stats(_np.asarray(d["gO"][cons][:, heads], _np.float64), Oc))
        lg = _np.asarray(d["gLSE"][heads][:, cons], _np.float64)
        l_st.append(_stats(lg, LSEc))
        rs = max(rs, float(_np.abs(_np.exp(LSEc - lg) - 1.0).max()))
    out["O"] = (max(x[0] for x in o_st), sum(x[1] for x in o_st), sum(x[2] for x in o_st))
    out["LSE"] = (max(x[0] for x in l_st), sum(x[1] for x in l_st), sum(x[2] for x in l_st))
    out["rowsum"] = rs
    out["rows_o"] = int(sum(len(c) for c, _, _ in fo.values()))
    dq = O.rows_dq(ti, d["Q"], d["K"], d["V"], d["dO"], scale, job["dq_rows"], heads)
    gq = _np.asarray(d["gdQ"][job["dq_rows"]][:, heads], _np.float64)
    out["dQ"] = _stats(gq, dq)
    if job["complete"]:
        sel = _np.isin(_np.asarray(job["dq_rows"]), _np.asarray(job["leaf_rows"]))
        out["dQ complete"] = _stats(gq[sel], dq[sel])
    return out


def check_full_size(wl, gpu, workers=8, tmpdir=None, gate=("O", "LSE", "dQ", "dK", "dV"), complete=True):
    """Element-by-element parity of the selected outputs of a full-size workload (see above);
    returns {tensor: (max-abs, rel-L2)} plus the counts checked.  Only the tensors in ``gate``
    (and their complete slices, when ``complete``) must meet the tolerances; the others are
    reported."""
    import multiprocessing as mp
    import shutil
    import tempfile
    Og, LSEg, dQg, dKg, dVg = gpu
    t = wl.tree
    ti, shared, leaf = _most_shared_and_leaf(t)
    keys = _tiles(int(t.row_off[shared]), int(t.seg_len[shared]), 128)
    if leaf != shared:
        keys = sorted(set(keys) | set(_tiles(int(t.row_off[leaf]), int(t.seg_len[leaf]), 128)))
    dq_rows = _tiles(int(t.row_off[shared]), int(t.seg_len[shared]), 64)
    if leaf != shared:
        dq_rows = sorted(set(dq_rows) | set(_tiles(int(t.row_off[leaf]), int(t.seg_len[leaf]), 64)))
    node_rows = lambda n: list(range(int(t.row_off[n]), int(t.row_off[n]) + int(t.seg_len[n])))
    keys_all = sorted(set(node_rows(shared)) | set(node_rows(leaf)))
    # the branch whose every dQ row is checked: the longest leaf of at most 1024 rows (else the
    # shortest), so that the per-row oracle stays within seconds
    leaves = [n for n in range(t.num_nodes) if not ti.children[n]]
    short = [n for n in leaves if int(t.seg_len[n]) <= 1024]
    branch = max(short, key=lambda n: (int(t.seg_len[n]), n)) if short else min(leaves, key=lambda n: (int(t.seg_len[n]), n))
    leaf_rows = node_rows(branch)
    tmp = tempfile.mkdtemp(prefix="psattn_parity_", dir=tmpdir)
    try:
        arrays = {"parent": t.parent, "seg_len": t.seg_len, "row_off": t.row_off, "row_slots": t.row_slots(),
                  "Q": wl.Q, "K": wl.K, "V": wl.V, "dO": wl.dO, "gO": Og.astype(np.float32),
                  "gLSE": LSEg.astype(np.float32), "gdQ": dQg.astype(np.float32), "gdK": dKg.astype(np.float32),
                  "gdV": dVg.astype(np.float32)}
        files = {}
        for k, v in arrays.items():
            files[k] = f"{tmp}/{k}.npy"
            np.save(files[k], np.ascontiguousarray(v))
        G = wl.hq // wl.hkv
        cores = len(os.sched_getaffinity(0))
        threads = max(1, cores // max(1, min(workers, wl.hkv)))
        jobs = [{"files": files, "g": g, "G": G, "scale": wl.scale, "keys": keys, "dq_rows": dq_rows,
                 "complete": False, "threads": threads} for g in range(wl.hkv)]
        if complete:   # the long job of the pool: more threads
            jobs[0].update(complete=True, keys=keys_all, dq_rows=sorted(set(dq_rows) | set(leaf_rows)),
                           leaf_rows=leaf_rows, threads=max(threads, cores // 2))
        env_keys = ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")
        saved = {k: os.environ.get(k) for k in env_keys}
        for k in env_keys:
            os.environ[k] = str(max(j["threads"] for j in jobs))
        try:
            with mp.get_context("spawn").Pool(min(workers, wl.hkv)) as pool:
                parts = pool.map(_full_size_worker, jobs)
        finally:
            for k, v in saved.items():
                if v is None:
                    os.environ.pop(k, None)
                else:
                    os.environ[k] = v
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    tau_abs, tau_rel = TOL[wl.dtype]
    res = {"keys": len(keys), "dq_rows": len(dq_rows), "o_rows": parts[0]["rows_o"], "shared_node": shared,
           "leaf": leaf}
    if complete:
        res.update({"keys complete": len(keys_all), "dq_rows complete": len(leaf_rows), "branch": branch})
    names = ["O", "LSE", "dQ", "dK", "dV"] + (["dQ complete", "dK complete", "dV complete"] if complete else [])
    for name in names:
        ps = [p[name] for p in parts if name in p]
        mx = max(x[0] for x in ps)
        num = sum(x[1] for x in ps)
        den = sum(x[2] for x in ps)
        rel = float(np.sqrt(num / den)) if den > 0 else float(np.sqrt(num))
        res[name] = (mx, rel)
    res["rowsum"] = max(p["rowsum"] for p in parts)
    for name in [n for n in names if n.split()[0] in gate]:
        mx, rel = res[name]
        assert mx <= tau_abs and rel <= tau_rel, f"{name}: max-abs {mx:.3g} (<= {tau_abs}), rel-L2 {rel:.3g} (<= {tau_rel})"
    assert res["rowsum"] <= ROWSUM_TOL[wl.dtype], f"softmax rows with the GPU LSE sum to 1 +- {res['rowsum']:.3g}"
    return res
