"""Pins of the oracle's decoder layer (oracle.layer / layer_sample), none of them comparing the
oracle with itself:

* central finite differences of the advantage-masked loss with respect to every input and weight
  element, on a tiny forest (the manual backward);
* torch autograd (fp64, CPU) of the same layer on one sequence, written with torch's own ops
  (rms_norm's formula, silu, and scaled_dot_product_attention for the attention);
* rotary embedding: identity at position 0, the inverse undoes it, pair norms kept, and a known
  value;
* forward-only reuse: the layer's output on a shared token is the same in every sample (checked
  inside oracle.layer), and the forest output equals each sample's own output.
"""
import numpy as np
import pytest

import oracle as O
from oracle import psattn_oracle as OM

torch = pytest.importorskip("torch")


def _weights(rng, H, hq, hkv, d, F):
    return {"g1": 1 + 0.1 * rng.standard_normal(H), "Wq": rng.standard_normal((H, hq * d)) / np.sqrt(H),
            "Wk": rng.standard_normal((H, hkv * d)) / np.sqrt(H), "Wv": rng.standard_normal((H, hkv * d)) / np.sqrt(H),
            "Wo": rng.standard_normal((hq * d, H)) / np.sqrt(hq * d), "g2": 1 + 0.1 * rng.standard_normal(H),
            "W1": rng.standard_normal((H, F)) / np.sqrt(H), "W3": rng.standard_normal((H, F)) / np.sqrt(H),
            "W2": rng.standard_normal((F, H)) / np.sqrt(F)}


def _forest(rng, H):
    parent, seg = [-1, 0, 0], [4, 3, 2]
    row_off = np.array([0, 4, 7])
    ends = [1, 2]
    X = rng.standard_normal((9, H))
    return parent, seg, row_off, ends, X


def _mask(s, idx):
    return (np.arange(len(idx)) % 2 == s % 2).astype(float)        # an interleaved per-sample mask


def _loss(parent, seg, row_off, ends, X, W, hq, hkv, scale, theta, eps, adv, c):
    # the loss itself, by running the expanded samples forward only
    total = 0.0
    for s, idx in enumerate(O.sample_rows(parent, seg, row_off, ends)):
        out, _, _ = OM.layer_sample(X[idx], np.arange(len(idx)), W, hq, hkv, scale, theta, eps,
                                    np.zeros((len(idx), X.shape[1])))
        total += adv[s] * np.sum(_mask(s, idx)[:, None] * out * c[None, :])
    return total


def test_layer_finite_differences():
    rng = np.random.default_rng(0)
    H, hq, hkv, d, F = 8, 2, 1, 4, 12
    W = _weights(rng, H, hq, hkv, d, F)
    parent, seg, row_off, ends, X = _forest(rng, H)
    adv, c = np.array([0.7, -1.3]), rng.standard_normal(H)
    args = (hq, hkv, 0.5, 50.0, 1e-6)
    out, dX, gW = O.layer(parent, seg, row_off, ends, X, W, *args, adv, _mask, c)
    f = lambda X_, W_: _loss(parent, seg, row_off, ends, X_, W_, *args, adv, c)
    hstep = 1e-6
    for i in np.ndindex(X.shape):
        Xp, Xm = X.copy(), X.copy()
        Xp[i] += hstep
        Xm[i] -= hstep
        fd = (f(Xp, W) - f(Xm, W)) / (2 * hstep)
        assert abs(fd - dX[i]) <= 1e-6 * max(1.0, abs(fd)), (i, fd, dX[i])
    for k in W:
        for i in np.ndindex(W[k].shape):
            Wp = {**W, k: W[k].copy()}
            Wm = {**W, k: W[k].copy()}
            Wp[k][i] += hstep
            Wm[k][i] -= hstep
            fd = (f(X, Wp) - f(X, Wm)) / (2 * hstep)
            assert abs(fd - gW[k][i]) <= 1e-6 * max(1.0, abs(fd)), (k, i, fd, gW[k][i])


def test_layer_matches_torch_autograd():
    import torch.nn.functional as F_
    rng = np.random.default_rng(1)
    H, hq, hkv, d, F, L = 32, 4, 2, 16, 48, 21
    W = _weights(rng, H, hq, hkv, d, F)
    x = rng.standard_normal((L, H))
    dout = rng.standard_normal((L, H))
    scale, theta, eps = 1 / np.sqrt(d), 10000.0, 1e-6
    out, dx, g = OM.layer_sample(x, np.arange(L), W, hq, hkv, scale, theta, eps, dout)
    T = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in W.items()}
    xt = torch.tensor(x, requires_grad=True)
    pos = torch.arange(L, dtype=torch.float64)
    inv = theta ** (-2.0 * torch.arange(d // 2, dtype=torch.float64) / d)
    ang = pos[:, None] * inv[None, :]
    cos, sin = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]

    def rope(t):
        a, b = t[..., : d // 2], t[..., d // 2:]
        return torch.cat([a * cos - b * sin, a * sin + b * cos], -1)

    rms = lambda t: t * torch.rsqrt(t.pow(2).mean(-1, keepdim=True) + eps)
    h = rms(xt) * T["g1"]
    q = rope((h @ T["Wq"]).view(L, hq, d)).permute(1, 0, 2)
    k = rope((h @ T["Wk"]).view(L, hkv, d)).permute(1, 0, 2).repeat_interleave(hq // hkv, 0)
    v = (h @ T["Wv"]).view(L, hkv, d).permute(1, 0, 2).repeat_interleave(hq // hkv, 0)
    o = F_.scaled_dot_product_attention(q, k, v, is_causal=True, scale=scale).permute(1, 0, 2).reshape(L, hq * d)
    y = xt + o @ T["Wo"]
    z = rms(y) * T["g2"]
    ot = y + (F_.silu(z @ T["W1"]) * (z @ T["W3"])) @ T["W2"]
    (ot * torch.tensor(dout)).sum().backward()
    assert np.max(np.abs(out - ot.detach().numpy())) <= 1e-10
    assert np.max(np.abs(dx - xt.grad.numpy())) <= 1e-10
    for kk in W:
        assert np.max(np.abs(g[kk] - T[kk].grad.numpy())) <= 1e-10, kk


def test_rope_pins():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, 3, 8))
    pos = np.array([0, 1, 7, 100, 4096])
    assert np.allclose(OM._rope(x[:1], pos[:1], 10000.0), x[:1], atol=0)
    y = OM._rope(x, pos, 10000.0)
    assert np.allclose(OM._rope(y, pos, 10000.0, -1.0), x, atol=1e-12)
    norm = lambda t: t[..., :4] ** 2 + t[..., 4:] ** 2
    assert np.allclose(norm(y), norm(x), atol=1e-12)
    e = np.zeros((1, 1, 2))
    e[0, 0, 0] = 1.0                                  # d = 2, pos 1, frequency 1: angle 1
    assert np.allclose(OM._rope(e, np.array([1]), 10000.0)[0, 0], [np.cos(1.0), np.sin(1.0)], atol=1e-15)


def test_forward_only_reuse_equals_each_sample():
    rng = np.random.default_rng(3)
    H, hq, hkv, d, F = 16, 2, 2, 8, 24
    W = _weights(rng, H, hq, hkv, d, F)
    parent, seg, row_off, ends, X = _forest(rng, H)
    out, _, _ = O.layer(parent, seg, row_off, ends, X, W, hq, hkv, 0.35, 10000.0, 1e-6, np.zeros(2), _mask,
                        np.zeros(H))
    for s, idx in enumerate(O.sample_rows(parent, seg, row_off, ends)):
        o_s, _, _ = OM.layer_sample(X[idx], np.arange(len(idx)), W, hq, hkv, 0.35, 10000.0, 1e-6,
                                    np.zeros((len(idx), H)))
        assert np.max(np.abs(out[idx] - o_s)) <= 1e-12
