"""One decoder layer over a prefix forest in the shared layout (Sec. 6, prefix-sharing training
runtime): every shared token is one row, computed once, whatever number of samples read it.

Forward (also the forward-only pass of the reference model and of the old-policy log-probs,
Sec. 6): h = rmsnorm(x) g1; q, k, v = h Wq, h Wk, h Wv; rotary embedding of q and k by each row's
sequence position (psattn_rope); k, v into their pool slots (psattn_kv_scatter); prefix-shared
attention (psattn_fwd); y = x + o Wo; z = rmsnorm(y) g2; out = y + (silu(z W1) * (z W3)) W2.

Backward: one pass over the accumulated adjoints (Sec. 6): the upstream gradient of a shared row
is the sum over the samples that read it (advantage_adjoint, Sec. 2.5 advantage masking), and the
layer's backward runs once on the shared rows (psattn_bwd for the attention, psattn_kv_gather and
the inverse rotation for its inputs).  The dense products are plain library GEMMs (torch on the
GPU); the tree-dependent steps are the library's kernels.
"""
from __future__ import annotations

from typing import Callable, Dict, Sequence, Tuple

import numpy as np

from . import psattn as P


def advantage_adjoint(parent, seg_len, row_off, sample_end, adv: Sequence[float],
                      loss_mask: Callable[[int, np.ndarray], np.ndarray], c: np.ndarray) -> np.ndarray:
    """Upstream gradient of every shared row for the loss sum_s A_s sum_t m_{s,t} <c, out_{s,t}>:
    row t collects A_s m_{s,t} c from every sample s whose path holds it (the earliest use of a
    shared token carries the loss terms of every later sample, Sec. 4.1.1).  loss_mask(s, rows)
    gives sample s's mask along its sequence (rows: the packed row of each position)."""
    parent = np.asarray(parent)
    seg_len = np.asarray(seg_len)
    row_off = np.asarray(row_off)
    ns = int(seg_len[row_off >= 0].sum())
    w = np.zeros(ns)
    for s, e in enumerate(sample_end):
        path = []
        n = int(e)
        while n >= 0:
            path.append(n)
            n = int(parent[n])
        rows = np.concatenate([np.arange(int(row_off[m]), int(row_off[m]) + int(seg_len[m])) for m in reversed(path)])
        w[rows] += float(adv[s]) * np.asarray(loss_mask(s, rows), dtype=np.float64)
    return w[:, None] * np.asarray(c, dtype=np.float64)[None, :]


class SharedLayer:
    """Weights W (torch tensors on the GPU, fp32 or bf16 like the tree): g1 [H], Wq [H, Hq d],
    Wk, Wv [H, Hkv d], Wo [Hq d, H], g2 [H], W1, W3 [H, F], W2 [F, H]."""

    def __init__(self, W: Dict[str, "torch.Tensor"], hq: int, hkv: int, head_dim: int, theta: float = 10000.0,
                 eps: float = 1e-6):
        self.W, self.hq, self.hkv, self.d, self.theta, self.eps = W, hq, hkv, head_dim, theta, eps

    def _rms(self, x):
        import torch
        return torch.rsqrt(x.float().pow(2).mean(-1, keepdim=True) + self.eps)

    def forward(self, tree: P.Tree, X, K_pool, V_pool):
        """out [Ns, H] and what the backward needs.  K_pool / V_pool receive this layer's K/V."""
        import torch
        W, ns, hq, hkv, d = self.W, tree.num_rows, self.hq, self.hkv, self.d
        dt = X.dtype
        r1 = self._rms(X)
        h = (X.float() * r1).to(dt) * W["g1"]
        q = (h @ W["Wq"]).view(ns, hq, d).contiguous()
        k = (h @ W["Wk"]).view(ns, hkv, d).contiguous()
        v = (h @ W["Wv"]).view(ns, hkv, d).contiguous()
        P.psattn_rope(tree, q, self.theta)
        P.psattn_rope(tree, k, self.theta)
        P.psattn_kv_scatter(tree, k, v, K_pool, V_pool)
        o_lo = torch.empty_like(q) if dt == torch.bfloat16 else None   # O's rounding residual (Delta)
        o, lse = P.psattn_fwd(tree, q, K_pool, V_pool, O_lo=o_lo)
        y = X + o.view(ns, hq * d) @ W["Wo"]
        r2 = self._rms(y)
        z = (y.float() * r2).to(dt) * W["g2"]
        a, b = z @ W["W1"], z @ W["W3"]
        m = torch.nn.functional.silu(a) * b
        out = y + m @ W["W2"]
        saved = dict(X=X, r1=r1, h=h, q=q, o=o, o_lo=o_lo, lse=lse, y=y, r2=r2, z=z, a=a, b=b, m=m, K=K_pool, V=V_pool)
        return out, saved

    def backward(self, tree: P.Tree, saved, dout):
        """dX [Ns, H] and the weight gradients for the summed upstream gradient dout [Ns, H]."""
        import torch
        W, ns, hq, hkv, d = self.W, tree.num_rows, self.hq, self.hkv, self.d
        s = saved
        f = lambda t: t.float()
        g = {}
        dout = f(dout)
        g["W2"] = f(s["m"]).t() @ dout
        dm = dout @ f(W["W2"]).t()
        a, b = f(s["a"]), f(s["b"])
        sig = torch.sigmoid(a)
        da = dm * b * (sig + a * sig * (1 - sig))
        db = dm * a * sig
        z = f(s["z"])
        g["W1"], g["W3"] = z.t() @ da, z.t() @ db
        dz = da @ f(W["W1"]).t() + db @ f(W["W3"]).t()
        yn = f(s["y"]) * s["r2"]
        g["g2"] = (dz * yn).sum(0)
        dzh = dz * f(W["g2"])
        dy = dout + (dzh - yn * (dzh * yn).mean(-1, keepdim=True)) * s["r2"]
        o = s["o"]
        g["Wo"] = f(o.view(ns, hq * d)).t() @ dy
        do = (dy @ f(W["Wo"]).t()).view(ns, hq, d).to(o.dtype).contiguous()
        dq, dKp, dVp = P.psattn_bwd(tree, s["q"], s["K"], s["V"], o, s["lse"], do, O_lo=s["o_lo"])
        dk, dv = P.psattn_kv_gather(tree, dKp, dVp)
        P.psattn_rope(tree, dq, self.theta, inverse=True)
        P.psattn_rope(tree, dk, self.theta, inverse=True)
        h = f(s["h"])
        dq2, dk2, dv2 = dq.view(ns, hq * d), dk.view(ns, hkv * d), dv.view(ns, hkv * d)
        g["Wq"], g["Wk"], g["Wv"] = h.t() @ dq2, h.t() @ dk2, h.t() @ dv2
        dh = dq2 @ f(W["Wq"]).t() + dk2 @ f(W["Wk"]).t() + dv2 @ f(W["Wv"]).t()
        xn = f(s["X"]) * s["r1"]
        g["g1"] = (dh * xn).sum(0)
        dhh = dh * f(W["g1"])
        dX = dy + (dhh - xn * (dhh * xn).mean(-1, keepdim=True)) * s["r1"]
        return dX, g
