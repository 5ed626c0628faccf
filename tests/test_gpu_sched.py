"""Eq. "single_sequence" fitted from GPU runs (Sec. 4.2: the coefficients come from profiling).

A call updates B sequences, each a suffix of l_suf new tokens after a cached prefix (an external
node, Sec. 4.1.1), so that a sequence's total length is l = prefix + l_suf.  The call's
forward + backward time on the GPU, divided by B, is one sample of T(l_suf, l); the host fit
(psattn_sched_fit) must explain the grid well and predict a held-out shape.  The fitted
coefficients are printed.
"""
import sys

import numpy as np
import pytest

from paper_2608_25683_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu, pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

B = 16                      # sequences per call: enough work items to fill the GPU
HQ, HKV, D = 32, 8, 128


def _per_sequence_ms(prefix, suffix, reps=7, warmup=2):
    from paper_2608_25683_amd import psattn as P
    parent, seg, ends, ext = [], [], [], []
    for _ in range(B):
        if prefix:
            parent += [-1, len(parent)]
            seg += [prefix, suffix]
            ext.append(len(parent) - 2)
        else:
            parent.append(-1)
            seg.append(suffix)
        ends.append(len(parent) - 1)
    wl = W.custom(parent, seg, ends, hq=HQ, hkv=HKV, d=D, dtype="bf16", tensors=False,
                  block_policy=lambda L: W.blocks_fixed(L, 64), shuffle_pool=False)
    call, _ = W.call_subset(wl, ends, ext)
    tree = P.Tree.from_workload(call, device="cuda")
    dev = torch.device("cuda")
    g = torch.Generator(device=dev).manual_seed(prefix * 7919 + suffix)
    ns, slots = call.tree.num_rows, call.tree.pool_slots

    def draw(shape):
        return (0.5 * torch.randn(shape, generator=g, device=dev)).to(torch.bfloat16)

    Q, dO = draw((ns, HQ, D)), draw((ns, HQ, D))
    K, V = draw((slots, HKV, D)), draw((slots, HKV, D))
    O_lo = torch.empty_like(Q)
    dK = torch.zeros((slots, HKV, D), dtype=torch.float32, device=dev)
    dV = torch.zeros_like(dK)
    times = []
    for r in range(warmup + reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        O, LSE = P.psattn_fwd(tree, Q, K, V, O_lo=O_lo)
        P.psattn_bwd(tree, Q, K, V, O, LSE, dO, dK=dK, dV=dV, O_lo=O_lo)
        e1.record()
        torch.cuda.synchronize()
        if r >= warmup:
            times.append(e0.elapsed_time(e1))
    return float(np.median(times)) / B


def test_cost_model_fitted_from_gpu_runs():
    from paper_2608_25683_amd import psattn as P
    grid = [(p, s) for p in (0, 1024, 2048) for s in (256, 512, 1024)]
    ls, ll, tt = [], [], []
    for p, s in grid:
        t = _per_sequence_ms(p, s)
        ls.append(s)
        ll.append(p + s)
        tt.append(t)
        print(f"prefix {p:5d} suffix {s:5d}: {t:.4f} ms per sequence", file=sys.stderr, flush=True)
    ls, ll, tt = (np.asarray(x, dtype=np.float64) for x in (ls, ll, tt))
    a = P.sched_fit(ls, ll, tt)
    pred = a[0] * ls * ll + a[1] * ls + a[2]
    r2 = 1.0 - np.sum((tt - pred) ** 2) / np.sum((tt - tt.mean()) ** 2)
    held = (1536, 384)
    t_held = _per_sequence_ms(*held)
    p_held = a[0] * held[1] * sum(held) + a[1] * held[1] + a[2]
    print(f"a1 {a[0]:.4g} ms/token^2, a2 {a[1]:.4g} ms/token, a3 {a[2]:.4g} ms; R^2 {r2:.4f}; held-out "
          f"{held}: measured {t_held:.4f}, predicted {p_held:.4f} ms", file=sys.stderr, flush=True)
    assert a[0] > 0
    assert r2 >= 0.95
    assert abs(p_held - t_held) <= 0.25 * t_held
