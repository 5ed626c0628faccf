"""One decoder layer in the shared layout on the GPU (Sec. 6): every shared token computed once,
one backward over the summed adjoints of an advantage-masked loss (Sec. 2.5), against the fp64
oracle that expands every sample and runs the layer on each independently (oracle.layer).

fp32 mode (true fp32 products everywhere, including the library GEMMs): the fp32 tolerance,
max-abs and relative L2 1e-5 per tensor, on the outputs, dX and every weight gradient (relative
to each tensor's largest entry for max-abs: weight gradients sum hundreds of rows).
"""
import sys

import numpy as np
import pytest

from paper_2608_25683_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

import oracle as O  # noqa: E402


def _mask(s, rows):
    return (np.arange(len(rows)) % 3 != s % 3).astype(float)      # a per-sample loss mask along the sequence


@pytest.mark.parametrize("hq,hkv,d", [(4, 2, 64), (8, 1, 128)])
def test_layer_matches_expanded_samples(hq, hkv, d):
    from paper_2608_25683_amd import psattn as P
    from paper_2608_25683_amd.layer import SharedLayer, advantage_adjoint
    wl = W.custom([-1, 0, 0, 1, -1], [90, 40, 25, 33, 50], [3, 2, 4], hq=hq, hkv=hkv, d=d, dtype="fp32", seed=51,
                  block_policy=lambda L: W.blocks_fixed(L, 16), tensors=False)
    t = wl.tree
    rng = np.random.default_rng(52)
    H, F = 96, 160
    Wn = {"g1": 1 + 0.1 * rng.standard_normal(H), "Wq": rng.standard_normal((H, hq * d)) / np.sqrt(H),
          "Wk": rng.standard_normal((H, hkv * d)) / np.sqrt(H), "Wv": rng.standard_normal((H, hkv * d)) / np.sqrt(H),
          "Wo": rng.standard_normal((hq * d, H)) / np.sqrt(hq * d), "g2": 1 + 0.1 * rng.standard_normal(H),
          "W1": rng.standard_normal((H, F)) / np.sqrt(H), "W3": rng.standard_normal((H, F)) / np.sqrt(H),
          "W2": rng.standard_normal((F, H)) / np.sqrt(F)}
    Wn = {k: v.astype(np.float32).astype(np.float64) for k, v in Wn.items()}
    X = rng.standard_normal((t.num_rows, H)).astype(np.float32).astype(np.float64)
    adv = np.array([1.5, -0.5, 0.8])
    c = rng.standard_normal(H).astype(np.float32).astype(np.float64)
    dev = torch.device("cuda")
    tree = P.Tree.from_workload(wl, device="cuda")
    layer = SharedLayer({k: torch.tensor(v, dtype=torch.float32, device=dev) for k, v in Wn.items()}, hq, hkv, d)
    Kp = torch.zeros((t.pool_slots, hkv, d), dtype=torch.float32, device=dev)
    Vp = torch.zeros_like(Kp)
    Xg = torch.tensor(X, dtype=torch.float32, device=dev)
    out, saved = layer.forward(tree, Xg, Kp, Vp)
    dout = advantage_adjoint(t.parent, t.seg_len, t.row_off, t.sample_end, adv, _mask, c)
    dX, g = layer.backward(tree, saved, torch.tensor(dout, dtype=torch.float32, device=dev))
    torch.cuda.synchronize()
    ref_out, ref_dX, ref_g = O.layer(t.parent, t.seg_len, t.row_off, t.sample_end, X, Wn, hq, hkv, wl.scale, 10000.0,
                                     1e-6, adv, _mask, c)
    res = {}
    for name, gv, rv in [("out", out, ref_out), ("dX", dX, ref_dX)] + [(k, g[k], ref_g[k]) for k in Wn]:
        gv = gv.double().cpu().numpy()
        err = np.abs(gv - rv)
        mx = float(err.max() / max(1.0, np.abs(rv).max()))
        rel = float(np.linalg.norm(gv - rv) / np.linalg.norm(rv))
        res[name] = (mx, rel)
        assert mx <= 1e-5 and rel <= 1e-5, f"{name}: max-abs {mx:.3g} rel-L2 {rel:.3g}"
    print(f"layer hq={hq} hkv={hkv} d={d}: {res}", file=sys.stderr)
