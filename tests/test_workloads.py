"""Pins of the seeded workload generator (exact integers per seed) and of bf16 rounding."""
import numpy as np
import pytest

from paper_2608_25683_amd import workloads as W

# name: (nodes, samples, blocks, pool_slots, Ns, Nu, max_sample, sum_nvis, K or None)
PINS = {
    "c1": (5, 4, 24, 384, 384, 768, 192, 49_344, None),
    "c2": (17, 16, 320, 20_480, 20_480, 81_920, 5_120, 83_896_320, None),
    # 256 branches of 16 on a 4096-token root, blocks of 16: sum_nvis = 4096*4097/2 + 256*(16*4096 + 136)
    "c2-small": (257, 256, 512, 8_192, 8_192, 1_052_672, 4_112, 25_202_688, None),
    "c3": (64, 64, 389, 41_552, 40_998, 187_643, 5_901, 105_901_670, None),
    "c4": (85, 64, 1_099, 46_112, 42_109, 219_694, 4_100, 126_438_093, None),
    "c5": (127, 127, 127, 107_703, 107_703, 234_026, 7_192, 202_132_990, 2),
}


@pytest.mark.parametrize("name", sorted(PINS))
def test_structural_pins(name):
    tree, extra = W.make_tree(name)
    s = W.tree_stats(tree, W.CONFIGS[name][1], W.CONFIGS[name][3])
    nodes, samples, blocks, slots, ns, nu, mx, nvis, K = PINS[name]
    assert (s["nodes"], s["samples"], s["blocks"], s["pool_slots"]) == (nodes, samples, blocks, slots)
    assert (s["Ns"], s["Nu"], s["max_sample"], s["sum_nvis"]) == (ns, nu, mx, nvis)
    if K is not None:
        assert extra["K"] == K


def test_ratio_pins():
    pmr = {"c2": 0.800, "c3": 0.975, "c4": 0.857, "c5": 0.742}
    red = {"c2": 0.750, "c3": 0.782, "c4": 0.808, "c5": 0.540}
    for name in pmr:
        tree, _ = W.make_tree(name)
        s = W.tree_stats(tree, 32, 128)
        assert round(s["pmr"], 3) == pmr[name]
        assert round(s["redundancy"], 3) == red[name]


def test_c5_segment_range_and_flops():
    tree, _ = W.make_tree("c5")
    s = W.tree_stats(tree, 40, 128)
    assert (s["min_seg"], s["max_seg"]) == (27, 5_134)
    # F_alg = 14 d Hq sum_nvis
    assert s["flop_alg"] == 14 * 128 * 40 * 202_132_990


def test_c2_flops_pin():
    tree, _ = W.make_tree("c2")
    assert W.tree_stats(tree, 32, 128)["flop_alg"] == 4_810_950_574_080


def test_chunked_draws_equal_one_draw():
    a = W._draw(np.random.default_rng(7), (1000, 3), 0.5, "bf16", chunk=97)
    b = W._draw(np.random.default_rng(7), (1000, 3), 0.5, "bf16", chunk=1 << 20)
    assert np.array_equal(a, b)


def test_bf16_rounding_is_nearest_even():
    # exact ties and near-ties around 1.0 (bf16 ulp at 1.0 is 2^-7)
    ulp = 2.0 ** -7
    x = np.array([1.0 + ulp / 2, 1.0 + 1.5 * ulp, 1.0 + ulp / 2 + 2.0 ** -40, -1.0 - ulp / 2,
                  1.0 + ulp / 2 - 2.0 ** -40, 3.0, 0.0, 9984.0, 1e4])
    got = W.round_to_bf16(x)
    want = np.array([1.0, 1.0 + 2 * ulp, 1.0 + ulp, -1.0, 1.0, 3.0, 0.0, 9984.0, 9984.0], dtype=np.float32)
    assert np.array_equal(got, want)
    # agrees with the fp32 -> bf16 round-to-nearest-even of torch for fp32-exact inputs
    torch = pytest.importorskip("torch")
    r = np.random.default_rng(0).standard_normal(100_000).astype(np.float32).astype(np.float64)
    ref = torch.tensor(r, dtype=torch.float32).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(W.round_to_bf16(r), ref)


def test_pool_scatter_and_sentinel():
    wl = W.make("c1")
    t = wl.tree
    slots = t.row_slots()
    assert len(np.unique(slots)) == t.num_rows
    assert np.array_equal(wl.K_pool[slots], wl.K)
    pad = np.setdiff1d(np.arange(t.pool_slots), slots)
    assert np.all(wl.K_pool[pad] == W.SENTINEL)


def test_block_policies():
    assert W.blocks_greedy(300) == [(256, 256), (16, 16), (16, 16), (16, 12)]
    assert W.blocks_greedy(1000) == [(256, 256)] * 3 + [(64, 64)] * 3 + [(16, 16), (16, 16), (16, 8)]
    assert W.blocks_fixed(70, 32) == [(32, 32), (32, 32), (32, 6)]
    assert W.blocks_exact(27) == [(27, 27)]
