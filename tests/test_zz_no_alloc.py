"""psattn_bwd_noalloc (the backward pass with its workspace in the library's per-GPU device array)
against psattn_bwd, through the C ABI: bitwise-equal outputs on two calls in a row, the second on a
smaller tree, and the size limit enforced before anything is enqueued."""
import pytest

from paper_2608_25683_amd import workloads as W

torch = pytest.importorskip("torch")
# torch's HIP runtime starts before the library is loaded (as in the other GPU test modules)
HAS_GPU = torch.cuda.is_available()
P = pytest.importorskip("paper_2608_25683_amd.psattn")


def test_noalloc_rejects_a_workspace_beyond_its_array():
    # 64 roots of 512 rows x 272 query heads: 4 statistics of 4 bytes per (row, head) are 136 MiB,
    # more than the 128 MiB array; rejected before any device call (no GPU needed)
    wl = W.custom([-1] * 64, [512] * 64, list(range(64)), hq=272, hkv=8, d=128, tensors=False,
                  block_policy=W.blocks_exact)
    tree = P.Tree.from_workload(wl)
    assert tree.workspace_size(1) > (P.NOALLOC_SCRATCH_MIB << 20)
    null = [None] * 10
    st = P.lib().psattn_bwd_noalloc(tree.handle, *null, None)
    assert P.STATUS[st] == "PSATTN_E_WORKSPACE"
    assert b"psattn_bwd_noalloc holds" in P.lib().psattn_last_error()


@pytest.mark.gpu
@pytest.mark.skipif(not HAS_GPU, reason="needs a GPU")
def test_noalloc_matches_bwd_on_two_calls():
    big = W.random_forest(901, max_nodes=9, max_seg=300, hq=8, hkv=2, d=128, dtype="bf16")
    small = W.custom([-1, 0, 0], [70, 33, 12], [1, 2], hq=4, hkv=1, d=64, dtype="bf16", seed=9,
                     block_policy=lambda L: W.blocks_fixed(L, 16))
    opts = [{"fwd_kv_split": 128, "bwd_q_chunk": 64}, None]   # the first call fills partial tiles and rows
    sizes = []
    for wl, o in zip((big, small), opts):
        tree = P.Tree.from_workload(wl, opts=o, device="cuda")
        sizes.append(tree.workspace_size(1))
        dev = torch.device("cuda")
        Q, K, V, dO = (torch.from_numpy(x).to(dev).to(torch.bfloat16) for x in (wl.Q, wl.K_pool, wl.V_pool, wl.dO))
        O_lo = torch.empty_like(Q)
        Og, LSEg = P.psattn_fwd(tree, Q, K, V, O_lo=O_lo)
        ref = P.psattn_bwd(tree, Q, K, V, Og, LSEg, dO, O_lo=O_lo)
        out = [torch.full_like(x, float("nan")) for x in ref]
        P.psattn_bwd_noalloc(tree, Q, K, V, Og, LSEg, dO, *out, O_lo=O_lo)
        torch.cuda.synchronize()
        for name, a, b in zip(("dQ", "dK", "dV"), ref, out):
            assert torch.equal(a, b), f"{name}: psattn_bwd_noalloc differs from psattn_bwd"
    assert sizes[1] < sizes[0]
