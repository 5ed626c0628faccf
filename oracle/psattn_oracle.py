"""fp64 CPU oracle for prefix-shared causal attention (TEST INFRASTRUCTURE ONLY).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this module.  The product path (the HIP library and its Python
binding) never imports, calls or links it, and it shares no code with them.

What it computes, written from the paper's correctness contract:

* Sec. 2.5 ("Attention Masking"): although Q/K/V of a shared prefix are
  stored once, each token attends only along the autoregressive dependency
  of its own sequence, so the shared result must equal what independent
  computation gives.  The plain definition is therefore: expand every
  sample into its full, unshared root-to-endpoint sequence, and run ordinary
  causal softmax attention on it.
* Sec. 6 (training runtime): gradient adjoints of all consumers of a shared
  prefix are accumulated on the shared representation, then one backward
  pass runs.  The adjoint handed in for a shared token (dO) is the total over
  its consumers (Sec. 4.1.1: the earliest micro-batch carries the loss of
  later sequences on the shared prefix).  The oracle gives that total to the
  token's *owner* -- the first sample, in sample order, whose path holds it --
  and zero to every other copy, runs the textbook attention backward per
  sample, and sums the gradients of all copies of each token.

Conventions (the paper is silent on these): softmax scale is a parameter
(1/sqrt(d) in the workloads); LSE is the natural log of the softmax
denominator; query head h reads key/value head h // G with G = Hq / Hkv.

Parity unpinned: nothing -- every function here is pinned by the CPU tests
(finite differences, closed forms, torch SDPA special cases, gradient
identities, dO-split invariance, agreement of the per-row/per-key
evaluators with the expanded oracle).
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

ROW_CHUNK = 512


# ----------------------------------------------------------------------------- tree helpers

def node_paths(parent: Sequence[int]) -> List[List[int]]:
    """Root-to-node list of node ids for every node."""
    paths: List[List[int]] = []
    for i, p in enumerate(parent):
        p = int(p)
        paths.append([i] if p < 0 else paths[p] + [i])
    return paths


def node_offsets(parent: Sequence[int], seg_len: Sequence[int]) -> np.ndarray:
    off = np.zeros(len(parent), dtype=np.int64)
    for i, p in enumerate(parent):
        p = int(p)
        off[i] = 0 if p < 0 else off[p] + int(seg_len[p])
    return off


def sample_rows(parent, seg_len, row_off, sample_end) -> List[np.ndarray]:
    """For each sample, the packed row index of every token of its unshared sequence."""
    paths = node_paths(parent)
    out = []
    for e in sample_end:
        idx = [np.arange(int(row_off[n]), int(row_off[n]) + int(seg_len[n])) for n in paths[int(e)]]
        out.append(np.concatenate(idx).astype(np.int64))
    return out


def owners(parent, sample_end) -> np.ndarray:
    """Owner sample of each node: the first sample in sample order whose path contains it."""
    paths = node_paths(parent)
    own = np.full(len(parent), -1, dtype=np.int64)
    for s, e in enumerate(sample_end):
        for n in paths[int(e)]:
            if own[n] < 0:
                own[n] = s
    return own


# ----------------------------------------------------------------------------- dense causal attention

def causal_fwd(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """Causal softmax attention of one sequence and one head, fp64.

    q, k, v: [L, d].  Row i sees keys 0..i.  Returns o [L, d] and
    lse [L] = log sum_j exp(scale * q_i . k_j), computed with the row max
    subtracted.
    """
    L = q.shape[0]
    o = np.empty_like(q, dtype=np.float64)
    lse = np.empty(L, dtype=np.float64)
    for c0 in range(0, L, ROW_CHUNK):
        c1 = min(L, c0 + ROW_CHUNK)
        s = scale * (q[c0:c1] @ k[:c1].T)                      # [rows, keys<=c1-1]
        mask = np.arange(c1)[None, :] > np.arange(c0, c1)[:, None]
        s[mask] = -np.inf
        m = s.max(axis=1, keepdims=True)
        e = np.exp(s - m)
        den = e.sum(axis=1, keepdims=True)
        lse[c0:c1] = (m + np.log(den))[:, 0]
        o[c0:c1] = (e / den) @ v[:c1]
    return o, lse


def causal_bwd(q, k, v, o, lse, do, scale) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Backward of :func:`causal_fwd` for upstream gradient ``do`` (fp64).

    With P = softmax(scale * Q K^T) under the causal mask:
      dV = P^T dO;  dP = dO V^T;  Delta_i = sum_d dO_i * O_i;
      dS = P * (dP - Delta);  dQ = scale * dS K;  dK = scale * dS^T Q.
    """
    L = q.shape[0]
    dq = np.zeros_like(q, dtype=np.float64)
    dk = np.zeros_like(k, dtype=np.float64)
    dv = np.zeros_like(v, dtype=np.float64)
    delta = np.sum(do * o, axis=1)
    for c0 in range(0, L, ROW_CHUNK):
        c1 = min(L, c0 + ROW_CHUNK)
        s = scale * (q[c0:c1] @ k[:c1].T)
        mask = np.arange(c1)[None, :] > np.arange(c0, c1)[:, None]
        p = np.exp(s - lse[c0:c1, None])
        p[mask] = 0.0
        dv[:c1] += p.T @ do[c0:c1]
        dp = do[c0:c1] @ v[:c1].T
        ds = p * (dp - delta[c0:c1, None])
        dq[c0:c1] = scale * (ds @ k[:c1])
        dk[:c1] += scale * (ds.T @ q[c0:c1])
    return dq, dk, dv


# ----------------------------------------------------------------------------- the expanded oracle

def _as64(x):
    return np.asarray(x, dtype=np.float64)


def forward(parent, seg_len, row_off, sample_end, Q, K, V, scale, check_copies=True, tol=1e-9):
    """Shared forward result, node-packed: O [Ns, Hq, d] and LSE [Hq, Ns] (fp64).

    Each sample is expanded and run independently; a shared token's output
    is its value in any sample containing it.  With ``check_copies`` every
    copy is compared and a mismatch beyond ``tol`` raises (shared == unshared).
    """
    Ns, Hq, d = Q.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    O = np.full((Ns, Hq, d), np.nan)
    LSE = np.full((Hq, Ns), np.nan)
    seen = np.zeros(Ns, dtype=bool)
    for rows in sample_rows(parent, seg_len, row_off, sample_end):
        for h in range(Hq):
            o, lse = causal_fwd(_as64(Q[rows, h]), _as64(K[rows, h // G]), _as64(V[rows, h // G]), scale)
            old = seen[rows]
            if check_copies and old.any():
                r_old = rows[old]
                err = max(np.max(np.abs(O[r_old, h] - o[old])), np.max(np.abs(LSE[h, r_old] - lse[old])))
                if err > tol:
                    raise AssertionError(f"shared != unshared: copies differ by {err}")
            O[rows, h] = o
            LSE[h, rows] = lse
        seen[rows] = True
    return O, LSE


def backward(parent, seg_len, row_off, sample_end, Q, K, V, dO, scale, split: str = "owner"):
    """Gradients of the shared inputs, node-packed, fp64: dQ [Ns,Hq,d], dK, dV [Ns,Hkv,d].

    ``dO`` is the total adjoint of each shared token.  ``split`` decides how
    it is handed to the copies: "owner" gives all of it to the first sample
    containing the token; "uniform" gives each of the r copies dO / r.  The
    result must not depend on the split.
    """
    Ns, Hq, d = Q.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    dQ = np.zeros((Ns, Hq, d))
    dK = np.zeros((Ns, Hkv, d))
    dV = np.zeros((Ns, Hkv, d))
    srows = sample_rows(parent, seg_len, row_off, sample_end)
    if split == "owner":
        own = owners(parent, sample_end)
        row_owner = np.empty(Ns, dtype=np.int64)
        for n in range(len(parent)):
            row_owner[int(row_off[n]):int(row_off[n]) + int(seg_len[n])] = own[n]
    elif split == "uniform":
        copies = np.zeros(Ns, dtype=np.int64)
        for rows in srows:
            copies[rows] += 1
    else:
        raise ValueError(split)
    for s, rows in enumerate(srows):
        if split == "owner":
            w = (row_owner[rows] == s).astype(np.float64)
        else:
            w = 1.0 / copies[rows]
        for h in range(Hq):
            q, k, v = _as64(Q[rows, h]), _as64(K[rows, h // G]), _as64(V[rows, h // G])
            o, lse = causal_fwd(q, k, v, scale)
            do = _as64(dO[rows, h]) * w[:, None]
            dq, dk, dv = causal_bwd(q, k, v, o, lse, do, scale)
            np.add.at(dQ, (rows, h), dq)
            np.add.at(dK, (rows, h // G), dk)
            np.add.at(dV, (rows, h // G), dv)
    return dQ, dK, dV


# ----------------------------------------------------------------------------- point evaluators
# The same definitions evaluated for selected outputs only, so that outputs of
# full-size workloads can be checked one by one.  Written in the shared form:
# a token of node n at position a sees every token of n's strict ancestors and
# the tokens 0..a of n; dO is the total adjoint.  The CPU tests pin these to
# the expanded oracle above.

class TreeIndex:
    def __init__(self, parent, seg_len, row_off):
        self.parent = np.asarray(parent, dtype=np.int64)
        self.seg_len = np.asarray(seg_len, dtype=np.int64)
        self.row_off = np.asarray(row_off, dtype=np.int64)
        n = len(self.parent)
        self.paths = node_paths(self.parent)
        self.off = node_offsets(self.parent, self.seg_len)
        self.row_node = np.empty(int(self.seg_len.sum()), dtype=np.int64)
        for i in range(n):
            self.row_node[self.row_off[i]:self.row_off[i] + self.seg_len[i]] = i
        self.children: List[List[int]] = [[] for _ in range(n)]
        for i, p in enumerate(self.parent):
            if p >= 0:
                self.children[int(p)].append(i)

    def path_rows(self, n: int) -> np.ndarray:
        return np.concatenate([np.arange(self.row_off[m], self.row_off[m] + self.seg_len[m]) for m in self.paths[n]])

    def subtree(self, n: int) -> List[int]:
        out, stack = [], [n]
        while stack:
            m = stack.pop()
            out.append(m)
            stack.extend(self.children[m])
        return sorted(out)


def rows_forward(ti: TreeIndex, Q, K, V, scale, rows: Sequence[int], heads: Sequence[int]):
    """O [len(rows), len(heads), d] and LSE [len(heads), len(rows)] of selected rows (fp64)."""
    Hq, Hkv = Q.shape[1], K.shape[1]
    G = Hq // Hkv
    rows = np.asarray(rows, dtype=np.int64)
    heads = list(heads)
    d = Q.shape[2]
    O = np.empty((len(rows), len(heads), d))
    LSE = np.empty((len(heads), len(rows)))
    by_node: Dict[int, List[int]] = {}
    for i, r in enumerate(rows):
        by_node.setdefault(int(ti.row_node[r]), []).append(i)
    for n, idx in by_node.items():
        idx = np.asarray(idx)
        prow = ti.path_rows(n)
        qpos = ti.off[n] + (rows[idx] - ti.row_off[n])            # sequence position of each query
        for c0 in range(0, len(idx), ROW_CHUNK):
            sel = idx[c0:c0 + ROW_CHUNK]
            qp = qpos[c0:c0 + ROW_CHUNK]
            nk = int(qp.max()) + 1
            mask = np.arange(nk)[None, :] > qp[:, None]
            for hi, h in enumerate(heads):
                q = _as64(Q[rows[sel], h])
                k = _as64(K[prow[:nk], h // G])
                v = _as64(V[prow[:nk], h // G])
                s = scale * (q @ k.T)
                s[mask] = -np.inf
                m = s.max(axis=1, keepdims=True)
                e = np.exp(s - m)
                den = e.sum(axis=1, keepdims=True)
                LSE[hi, sel] = (m + np.log(den))[:, 0]
                O[sel, hi] = (e / den) @ v
    return O, LSE


def rows_dq(ti: TreeIndex, Q, K, V, dO, scale, rows: Sequence[int], heads: Sequence[int]):
    """dQ [len(rows), len(heads), d] of selected rows: scale * sum_j P_ij (dP_ij - Delta_i) k_j."""
    Hq, Hkv = Q.shape[1], K.shape[1]
    G = Hq // Hkv
    rows = np.asarray(rows, dtype=np.int64)
    O, LSE = rows_forward(ti, Q, K, V, scale, rows, heads)
    out = np.empty_like(O)
    for i, r in enumerate(rows):
        n = int(ti.row_node[r])
        nk = int(ti.off[n] + (r - ti.row_off[n])) + 1
        prow = ti.path_rows(n)[:nk]
        for hi, h in enumerate(heads):
            q = _as64(Q[r, h])
            k = _as64(K[prow, h // G])
            v = _as64(V[prow, h // G])
            do = _as64(dO[r, h])
            p = np.exp(scale * (k @ q) - LSE[hi, i])
            dp = v @ do
            delta = float(do @ O[i, hi])
            out[i, hi] = scale * ((p * (dp - delta)) @ k)
    return out


def keys_dkdv(ti: TreeIndex, Q, K, V, dO, scale, key_rows: Sequence[int], kv_head: int, forward_out=None):
    """dK, dV [len(key_rows), d] of selected key rows for one kv head (fp64).

    Consumers of key row j (node m, position b) are rows of m at positions
    >= b and every row of every descendant of m; each consumer contributes
    through all G query heads that read kv head ``kv_head``.  If
    ``forward_out`` is a dict, the consumers' forward results are left in it:
    forward_out[m] = (consumer rows, O [rows, G, d], LSE [G, rows]).
    """
    Hq, Hkv = Q.shape[1], K.shape[1]
    G = Hq // Hkv
    heads = list(range(kv_head * G, (kv_head + 1) * G))
    key_rows = np.asarray(key_rows, dtype=np.int64)
    d = Q.shape[2]
    dK = np.zeros((len(key_rows), d))
    dV = np.zeros((len(key_rows), d))
    # consumers of all selected keys, grouped by the key's node
    by_node: Dict[int, List[int]] = {}
    for i, j in enumerate(key_rows):
        by_node.setdefault(int(ti.row_node[j]), []).append(i)
    for m, kidx in by_node.items():
        bmin = int(min(key_rows[kidx] - ti.row_off[m]))
        cons = [np.arange(ti.row_off[m] + bmin, ti.row_off[m] + ti.seg_len[m])]
        for c in ti.subtree(m):
            if c != m:
                cons.append(np.arange(ti.row_off[c], ti.row_off[c] + ti.seg_len[c]))
        cons = np.concatenate(cons)
        O, LSE = rows_forward(ti, Q, K, V, scale, cons, heads)
        if forward_out is not None:
            forward_out[m] = (cons, O, LSE)
        qpos = ti.off[ti.row_node[cons]] + (cons - ti.row_off[ti.row_node[cons]])
        kidx = np.asarray(kidx)
        kpos = ti.off[m] + (key_rows[kidx] - ti.row_off[m])
        vis = qpos[:, None] >= kpos[None, :]                        # [consumers, keys]
        kj = _as64(K[key_rows[kidx], kv_head])                       # [keys, d]
        vj = _as64(V[key_rows[kidx], kv_head])
        for hi, h in enumerate(heads):
            q = _as64(Q[cons, h])
            do = _as64(dO[cons, h])
            s = np.where(vis, scale * (q @ kj.T), -np.inf)
            p = np.exp(s - LSE[hi][:, None])                         # P_ij of every consumer i, key j
            dp = do @ vj.T                                           # dP_ij = dO_i . v_j
            delta = np.sum(do * O[:, hi], axis=1)                    # Delta_i = dO_i . O_i
            dV[kidx] += p.T @ do
            dK[kidx] += scale * ((p * (dp - delta[:, None])).T @ q)
    return dK, dV


# ----------------------------------------------------------------------------- one decoder layer
#
# The rest of a layer, written the same plain way: every sample expanded into its own sequence
# and run through one decoder layer independently, gradients of duplicated tokens summed (Sec.
# 2.5: shared results equal independent computation; Sec. 6: one backward over the accumulated
# adjoints).  The layer: h = rmsnorm(x) g1; q, k, v = h Wq, h Wk, h Wv; rotary embedding of q and
# k by sequence position; causal attention; y = x + o Wo; z = rmsnorm(y) g2;
# out = y + (silu(z W1) * (z W3)) W2.  The loss of sample s is advantage-masked (Sec. 2.5):
# L_s = A_s * sum_t m_{s,t} <c, out_{s,t}>, so each token counts only for the samples whose mask
# holds it.

def _rms(x, eps):
    return np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def _rope(x, pos, theta, sign=1.0):
    """x [L, heads, d]: pairs (i, i + d/2) turned by sign * pos * theta^(-2i/d)."""
    d = x.shape[-1]
    half = d // 2
    ang = sign * pos[:, None].astype(np.float64) * theta ** (-2.0 * np.arange(half) / d)[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def layer_sample(x, pos, W, hq, hkv, scale, theta, eps, dout):
    """One decoder layer on one sequence (fp64) and its backward for upstream gradient dout.

    x [L, H]; pos [L]; W: g1, Wq, Wk, Wv, Wo, g2, W1, W3, W2.  Returns out [L, H], dx [L, H] and
    the weight gradients (dict).
    """
    L = x.shape[0]
    d = W["Wq"].shape[1] // hq
    G = hq // hkv
    r1 = _rms(x, eps)
    h = x / r1 * W["g1"]
    q = _rope((h @ W["Wq"]).reshape(L, hq, d), pos, theta)
    k = _rope((h @ W["Wk"]).reshape(L, hkv, d), pos, theta)
    v = (h @ W["Wv"]).reshape(L, hkv, d)
    o = np.empty((L, hq, d))
    lse = np.empty((hq, L))
    for j in range(hq):
        o[:, j], lse[j] = causal_fwd(q[:, j], k[:, j // G], v[:, j // G], scale)
    y = x + o.reshape(L, hq * d) @ W["Wo"]
    r2 = _rms(y, eps)
    z = y / r2 * W["g2"]
    a, b = z @ W["W1"], z @ W["W3"]
    sig = 1.0 / (1.0 + np.exp(-a))
    m = a * sig * b
    out = y + m @ W["W2"]
    # backward
    g = {}
    g["W2"] = m.T @ dout
    dm = dout @ W["W2"].T
    da = dm * b * (sig + a * sig * (1.0 - sig))
    db = dm * a * sig
    g["W1"], g["W3"] = z.T @ da, z.T @ db
    dz = da @ W["W1"].T + db @ W["W3"].T
    g["g2"] = np.sum(dz * y / r2, axis=0)
    dzh = dz * W["g2"]
    dy = dout + (dzh - (y / r2) * np.mean(dzh * y / r2, axis=-1, keepdims=True)) / r2
    g["Wo"] = o.reshape(L, hq * d).T @ dy
    do = (dy @ W["Wo"].T).reshape(L, hq, d)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for j in range(hq):
        a_q, a_k, a_v = causal_bwd(q[:, j], k[:, j // G], v[:, j // G], o[:, j], lse[j], do[:, j], scale)
        dq[:, j] += a_q
        dk[:, j // G] += a_k
        dv[:, j // G] += a_v
    dq = _rope(dq, pos, theta, -1.0).reshape(L, hq * d)
    dk = _rope(dk, pos, theta, -1.0).reshape(L, hkv * d)
    dv = dv.reshape(L, hkv * d)
    g["Wq"], g["Wk"], g["Wv"] = h.T @ dq, h.T @ dk, h.T @ dv
    dh = dq @ W["Wq"].T + dk @ W["Wk"].T + dv @ W["Wv"].T
    g["g1"] = np.sum(dh * x / r1, axis=0)
    dhh = dh * W["g1"]
    dx = dy + (dhh - (x / r1) * np.mean(dhh * x / r1, axis=-1, keepdims=True)) / r1
    return out, dx, g


def layer(parent, seg_len, row_off, sample_end, X, W, hq, hkv, scale, theta, eps, adv, loss_mask, c):
    """The layer over a prefix forest, by expansion (fp64).

    X [Ns, H] hidden state of every shared row; adv [S] advantage of each sample; loss_mask(s, rows)
    -> 0/1 per position of sample s's sequence; c [H] the loss direction.  Returns out [Ns, H]
    (checked equal on every copy of a shared token), dX [Ns, H] (duplicates summed) and the
    weight gradients summed over samples.
    """
    X = _as64(X)
    W = {k: _as64(v) for k, v in W.items()}
    off = node_offsets(parent, seg_len)
    out = np.full(X.shape, np.nan)
    dX = np.zeros_like(X)
    gW = {k: np.zeros_like(v) for k, v in W.items()}
    for s, idx in enumerate(sample_rows(parent, seg_len, row_off, sample_end)):
        pos = np.arange(len(idx))
        dout = float(adv[s]) * np.asarray(loss_mask(s, idx), dtype=np.float64)[:, None] * _as64(c)[None, :]
        o_s, dx_s, g_s = layer_sample(X[idx], pos, W, hq, hkv, scale, theta, eps, dout)
        seen = ~np.isnan(out[idx, 0])
        if np.any(seen):
            assert np.max(np.abs(out[idx][seen] - o_s[seen])) <= 1e-9, "copies of a shared token differ"
        out[idx] = o_s
        np.add.at(dX, idx, dx_s)
        for k in gW:
            gW[k] += g_s[k]
    return out, dX, gW
