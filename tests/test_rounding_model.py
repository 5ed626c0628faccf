"""Why the dK/dV products take P and dS as two bf16 terms: a CPU model of the rounding.

dV_j = sum_i P_ij dO_i and dK_j = scale sum_i dS_ij Q_i sum over every consumer i of key j (all
rows of all branches that reuse it, times the G query heads of its kv group).  If P and dS are
rounded once to bf16 before those products, each term carries a relative error of up to 2^-9 and
the errors add up like a random walk: ~2^-9/sqrt(3) * sqrt(sum_i P_ij^2 dO_i^2).  On a key that
many consumers weight heavily (40 one-token siblings at G = 5; an attention-sink-like root key)
that exceeds the 2e-2 max-abs bound.  With x = hi + lo (hi = bf16(x), lo = bf16(x - hi)) the
remaining error is ~2^-17 relative per term.

The model evaluates the exact P and dS of one key's consumers in fp64 (from the oracle's
per-row forward), applies each rounding, and sums in fp64, so the only error left is the
rounding of P and dS.
"""
import numpy as np
import pytest

import oracle as O
from paper_2608_25683_amd import workloads as W

TAU_ABS = 2e-2


def bf16(x):
    return W.round_to_bf16(np.asarray(x, dtype=np.float64)).astype(np.float64)


def two_term(x):
    hi = bf16(x)
    return hi + bf16(x - hi)


def key_errors(wl, key_row, kv_head):
    """max |error| of (dK, dV) of one key under each rounding of P and dS, and the consumer count."""
    t = wl.tree
    ti = O.TreeIndex(t.parent, t.seg_len, t.row_off)
    G = wl.hq // wl.hkv
    heads = list(range(kv_head * G, (kv_head + 1) * G))
    node = int(ti.row_node[key_row])
    kpos = ti.off[node] + (key_row - ti.row_off[node])
    cons = [r for r in range(t.num_rows)
            if node in ti.paths[int(ti.row_node[r])] and ti.off[ti.row_node[r]] + r - ti.row_off[ti.row_node[r]] >= kpos]
    cons = np.asarray(cons, dtype=np.int64)
    o, lse = O.rows_forward(ti, wl.Q, wl.K, wl.V, wl.scale, cons, heads)
    dk_ref, dv_ref = O.keys_dkdv(ti, wl.Q, wl.K, wl.V, wl.dO, wl.scale, [key_row], kv_head)
    Q, dO = wl.Q.astype(np.float64), wl.dO.astype(np.float64)
    k, v = wl.K[key_row, kv_head].astype(np.float64), wl.V[key_row, kv_head].astype(np.float64)
    out = {}
    for name, rnd in (("exact", lambda x: x), ("bf16", bf16), ("two_term", two_term)):
        dk = np.zeros_like(k)
        dv = np.zeros_like(v)
        for jh, h in enumerate(heads):
            p = np.exp(wl.scale * (Q[cons, h] @ k) - lse[jh])
            ds = p * (dO[cons, h] @ v - np.sum(dO[cons, h] * o[:, jh], axis=1))
            dv += rnd(p) @ dO[cons, h]
            dk += wl.scale * (rnd(ds) @ Q[cons, h])
        out[name] = (float(np.abs(dk - dk_ref[0]).max()), float(np.abs(dv - dv_ref[0]).max()))
    return len(cons) * G, out


def test_exact_model_matches_the_oracle():
    wl = W.custom([-1, 0, 0], [20, 7, 9], [1, 2], hq=4, hkv=2, d=64, dtype="bf16", seed=3,
                  block_policy=W.blocks_exact)
    _, e = key_errors(wl, 5, 1)
    assert max(e["exact"]) < 1e-12


def test_forty_one_token_siblings_at_g5():
    wl = W.custom([-1] + [0] * 40, [1] * 41, list(range(1, 41)), hq=5, hkv=1, d=128, dtype="bf16", seed=11,
                  block_policy=W.blocks_exact)
    n, e = key_errors(wl, 0, 0)
    assert n == 205
    assert e["bf16"][1] > TAU_ABS            # dV with a single rounding of P: over the bound
    assert max(e["two_term"]) < 2e-4         # the split holds it


@pytest.mark.parametrize("kv_head", [0, 1])
def test_attention_sink_root_key(kv_head):
    wl = W.custom([-1] + [0] * 32, [512] + [16] * 32, list(range(1, 33)), hq=8, hkv=2, d=128, dtype="bf16", seed=21,
                  block_policy=lambda L: W.blocks_fixed(L, 64))
    W.add_attention_sink(wl, [0], logit=float(np.log(528.0)))
    n, e = key_errors(wl, 0, kv_head)
    assert n == 4096
    assert e["bf16"][1] > 5 * TAU_ABS        # dV: several times the bound
    assert e["bf16"][0] > TAU_ABS            # dK too
    assert max(e["two_term"]) < 1e-3


def test_error_grows_like_sqrt_of_consumers():
    # one-token siblings under a one-token root, P on the root key near 1/2 for every sibling:
    # the single-rounding dV error follows sqrt(n) (mean over seeds), the split stays flat
    grow, flat = [], []
    for nsib in (16, 256):
        e1, e2 = [], []
        for seed in range(4):
            wl = W.custom([-1] + [0] * nsib, [1] * (nsib + 1), list(range(1, nsib + 1)), hq=4, hkv=1, d=64,
                          dtype="bf16", seed=100 + seed, block_policy=W.blocks_exact)
            _, e = key_errors(wl, 0, 0)
            e1.append(e["bf16"][1])
            e2.append(e["two_term"][1])
        grow.append(np.mean(e1))
        flat.append(np.mean(e2))
    ratio = grow[1] / grow[0]                # sqrt(256 / 16) = 4
    assert 2.0 < ratio < 8.0, grow
    assert flat[1] < grow[1] / 100
