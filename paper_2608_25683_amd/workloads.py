"""Seeded synthetic workloads: prefix trees, page tables and input tensors.

This module describes *inputs* only.  It draws trees shaped like the paper's
update-phase batches (tree sampling, step-wise sampling and tree-step
sampling, Sec. 2.3), lays the shared K/V rows out in a variable-block page
pool (one logical block per shared segment or fixed-size pages, Sec. 5.1 and
Fig. "Block_Management"), and draws Q/K/V/dO.  It contains no attention
arithmetic: both the fp64 oracle and the HIP path consume what it produces,
and neither is imported here.

Generator recipe (exact, so that the structural pins reproduce):

* ``rng_tree, rng_tensor = [default_rng(s) for s in SeedSequence(seed).spawn(2)]``
* nodes are appended in generation order (parents first); rows of the packed
  Q/O/dO/dQ/LSE tensors follow node order;
* tensors come from ``rng_tensor`` in the order Q(Ns,Hq,d), K(Ns,Hkv,d),
  V(Ns,Hkv,d), dO(Ns,Hq,d), all ``standard_normal`` float64; Q, K and V are
  scaled by ``sigma``; each is rounded once (round-to-nearest-even) to the
  config dtype;
* the page pool then places blocks in the order
  ``rng_tensor.permutation(num_blocks)``, each block taking ``capacity``
  consecutive slots; pad slots hold the sentinel bf16(1e4) = 9984.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence, Tuple

import numpy as np

SENTINEL = 9984.0  # bf16(1e4): large, finite, exactly representable in bf16 and fp32

# name -> (seed, hq, hkv, d, dtype, sigma, description)
CONFIGS = {
    "c1": (1, 4, 4, 64, "fp32", 1.0,
           "tiny tree, fp32: MHA 4 heads, d64; root 128 + 4 branches of 64; page block 16"),
    "c2": (2, 32, 8, 128, "bf16", 0.5,
           "Llama-3-8B-shaped GQA 32q/8kv d128 bf16; depth-1 tree: prefix 4096 + 16 branches of 1024; page block 64"),
    "c3": (3, 32, 8, 128, "bf16", 0.5,
           "step-wise RL chains, 32q/8kv d128 bf16: 8 trajectories x 8 steps of U[256,1024]; adaptive blocks {256,64,16}"),
    "c4": (4, 32, 8, 128, "bf16", 0.5,
           "tree sampling, 32q/8kv d128 bf16: root 2048, branching 4, depth 3 (64 leaves), segments U[128,768]; per-node block size"),
    "c2-small": (6, 32, 8, 128, "bf16", 0.5,
                 "small-suffix probe, Llama-3-8B-shaped GQA 32q/8kv d128 bf16: prefix 4096 + 256 branches of 16; page block 16"),
    "c5": (5, 40, 8, 128, "bf16", 0.5,
           "Qwen2.5-32B-shaped 40q/8kv d128 bf16: 32 trees depth 2-4, branching 2-6, log-normal segments; tree-step samples; exact-length blocks"),
}

C5_NU_BUDGET = 262144


@dataclasses.dataclass
class Tree:
    """A prefix forest plus its page table, in the layout the C ABI consumes."""
    parent: np.ndarray        # int32 [N]; parent[i] < i or -1
    seg_len: np.ndarray       # int32 [N]
    row_off: np.ndarray       # int64 [N]; first packed row of node i
    blk_ptr: np.ndarray       # int32 [N+1]; CSR into the block arrays, token order
    blk_base: np.ndarray      # int64 [B]; first pool slot of each block
    blk_cap: np.ndarray       # int32 [B]
    blk_len: np.ndarray       # int32 [B]
    blk_pos: np.ndarray       # int32 [B]; absolute sequence position of the block's first token
    pool_slots: int
    sample_end: np.ndarray    # int32 [S]; endpoint node of each sample

    @property
    def num_nodes(self) -> int:
        return int(self.parent.shape[0])

    @property
    def num_rows(self) -> int:
        """Query rows of this call: nodes with row_off < 0 are external (cached by an earlier call)."""
        return int(self.seg_len[self.row_off >= 0].sum())

    def node_offsets(self) -> np.ndarray:
        """Sum of ancestor segment lengths per node (the sequence position of its first token)."""
        off = np.zeros(self.num_nodes, dtype=np.int64)
        for i in range(self.num_nodes):
            p = int(self.parent[i])
            off[i] = 0 if p < 0 else off[p] + int(self.seg_len[p])
        return off

    def path(self, node: int) -> List[int]:
        out = []
        while node >= 0:
            out.append(node)
            node = int(self.parent[node])
        return out[::-1]

    def row_slots(self) -> np.ndarray:
        """Pool slot holding each packed row's K/V (int64 [Ns])."""
        slots = np.empty(self.num_rows, dtype=np.int64)
        for n in range(self.num_nodes):
            if self.row_off[n] < 0:
                continue
            t = int(self.row_off[n])
            for b in range(int(self.blk_ptr[n]), int(self.blk_ptr[n + 1])):
                ln = int(self.blk_len[b])
                slots[t:t + ln] = int(self.blk_base[b]) + np.arange(ln)
                t += ln
        return slots


@dataclasses.dataclass
class Workload:
    name: str
    tree: Tree
    hq: int
    hkv: int
    d: int
    dtype: str                # "bf16" or "fp32"
    scale: float
    Q: Optional[np.ndarray] = None     # float32 [Ns, Hq, d] (bf16-exact values in bf16 mode)
    K: Optional[np.ndarray] = None     # float32 [Ns, Hkv, d] node-packed
    V: Optional[np.ndarray] = None
    dO: Optional[np.ndarray] = None    # float32 [Ns, Hq, d]
    K_pool: Optional[np.ndarray] = None  # float32 [pool_slots, Hkv, d]
    V_pool: Optional[np.ndarray] = None

    def stats(self) -> dict:
        return tree_stats(self.tree, self.hq, self.d)


# --------------------------------------------------------------------------- rounding

def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values once, to nearest-even bf16; returned as float32 (exact)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    bits = x.view(np.uint64)
    tiny = (np.abs(x) < 2.0 ** -126) & (x != 0)
    if tiny.any():
        raise ValueError("bf16 rounding: subnormal input not supported")
    drop = np.uint64(45)  # 52 fraction bits in fp64, 7 in bf16
    lsb = (bits >> drop) & np.uint64(1)
    rounded = (bits + (np.uint64((1 << 44) - 1) + lsb)) & ~np.uint64((1 << 45) - 1)
    return rounded.view(np.float64).astype(np.float32)


def _round(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_to_bf16(x)
    if dtype == "fp32":
        return x.astype(np.float32)
    raise ValueError(dtype)


def _draw(rng: np.random.Generator, shape: Tuple[int, ...], sigma: float, dtype: str,
          chunk: int = 1 << 22) -> np.ndarray:
    """standard_normal(shape) * sigma rounded to dtype, drawn in chunks (same stream)."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        v = rng.standard_normal(e - s)
        if sigma != 1.0:
            v *= sigma
        out[s:e] = _round(v, dtype)
    return out.reshape(shape)


def _skip_draw(rng: np.random.Generator, n: int, chunk: int = 1 << 22) -> None:
    for s in range(0, n, chunk):
        rng.standard_normal(min(chunk, n - s))


# --------------------------------------------------------------------------- block policies

def blocks_fixed(seg_len: int, size: int) -> List[Tuple[int, int]]:
    """Fixed-size pages: (capacity, len) per block; the last may be partial."""
    out = []
    left = seg_len
    while left > 0:
        ln = min(size, left)
        out.append((size, ln))
        left -= ln
    return out


def blocks_greedy(seg_len: int, sizes: Sequence[int] = (256, 64, 16)) -> List[Tuple[int, int]]:
    """Largest-first decomposition; only the final block of the smallest size may be partial."""
    out = []
    left = seg_len
    for s in sizes[:-1]:
        while left >= s:
            out.append((s, s))
            left -= s
    s = sizes[-1]
    while left > 0:
        ln = min(s, left)
        out.append((s, ln))
        left -= ln
    return out


def blocks_exact(seg_len: int) -> List[Tuple[int, int]]:
    """Adaptive block allocation: one block sized exactly to the shared segment (Sec. 5.1)."""
    return [(seg_len, seg_len)]


# --------------------------------------------------------------------------- trees

def _make_tree(parent: Sequence[int], seg_len: Sequence[int], node_blocks: Sequence[List[Tuple[int, int]]],
               sample_end: Sequence[int], perm: Optional[np.ndarray] = None) -> Tree:
    n = len(parent)
    parent = np.asarray(parent, dtype=np.int32)
    seg_len = np.asarray(seg_len, dtype=np.int32)
    row_off = np.zeros(n, dtype=np.int64)
    if n > 1:
        row_off[1:] = np.cumsum(seg_len[:-1], dtype=np.int64)
    off = np.zeros(n, dtype=np.int64)
    for i in range(n):
        p = int(parent[i])
        off[i] = 0 if p < 0 else off[p] + seg_len[p]
    blk_ptr = np.zeros(n + 1, dtype=np.int32)
    caps, lens, poss = [], [], []
    for i in range(n):
        pos = int(off[i])
        for cap, ln in node_blocks[i]:
            caps.append(cap)
            lens.append(ln)
            poss.append(pos)
            pos += ln
        blk_ptr[i + 1] = len(caps)
    nb = len(caps)
    caps = np.asarray(caps, dtype=np.int32)
    order = np.arange(nb) if perm is None else np.asarray(perm)
    base = np.zeros(nb, dtype=np.int64)
    cur = 0
    for b in order:
        base[b] = cur
        cur += int(caps[b])
    return Tree(parent=parent, seg_len=seg_len, row_off=row_off, blk_ptr=blk_ptr,
                blk_base=base, blk_cap=caps, blk_len=np.asarray(lens, dtype=np.int32),
                blk_pos=np.asarray(poss, dtype=np.int32), pool_slots=int(cur),
                sample_end=np.asarray(sample_end, dtype=np.int32))


def _struct_c1(rng):
    parent = [-1] + [0] * 4
    seg = [128] + [64] * 4
    return parent, seg, [blocks_fixed(L, 16) for L in seg], [1, 2, 3, 4]


def _struct_c2(rng):
    parent = [-1] + [0] * 16
    seg = [4096] + [1024] * 16
    return parent, seg, [blocks_fixed(L, 64) for L in seg], list(range(1, 17))


def _struct_c2_small(rng):
    # few queries per branch against a long shared prefix: the gather-bound end of the path
    parent = [-1] + [0] * 256
    seg = [4096] + [16] * 256
    return parent, seg, [blocks_fixed(L, 16) for L in seg], list(range(1, 257))


def _struct_c3(rng):
    parent, seg = [], []
    for traj in range(8):
        prev = -1
        for step in range(8):
            L = int(rng.integers(256, 1025))
            parent.append(prev)
            seg.append(L)
            prev = len(seg) - 1
    return parent, seg, [blocks_greedy(L) for L in seg], list(range(len(seg)))


def _struct_c4(rng):
    parent, seg = [-1], [2048]
    level = [0]
    for _ in range(3):
        nxt = []
        for p in level:
            for _c in range(4):
                parent.append(p)
                seg.append(int(rng.integers(128, 769)))
                nxt.append(len(seg) - 1)
        level = nxt
    sizes = [int(rng.choice([16, 32, 64, 128, 256])) for _ in seg]
    blocks = [blocks_fixed(L, B) for L, B in zip(seg, sizes)]
    return parent, seg, blocks, level


def _ln512(rng) -> int:
    v = math.exp(float(rng.normal(math.log(512.0), 1.0)))
    return int(min(8192, max(16, int(np.round(v)))))


def _struct_c5(rng, budget: int = C5_NU_BUDGET):
    # generate 32 full trees; each tree: list of levels, each node (parent_local, L)
    trees = []
    for _t in range(32):
        D = int(rng.integers(2, 5))
        nodes = [(-1, _ln512(rng))]
        level = [0]
        for _lv in range(1, D):
            nxt = []
            for p in level:
                b = int(rng.integers(2, 7))
                for _c in range(b):
                    nodes.append((p, _ln512(rng)))
                    nxt.append(len(nodes) - 1)
            level = nxt
        trees.append((nodes, level))

    def prune(nodes, leaves, k):
        keep = set()
        for leaf in leaves[:k]:
            n = leaf
            while n >= 0 and n not in keep:
                keep.add(n)
                n = nodes[n][0]
        return sorted(keep)

    def nu_for(k):
        tot = 0
        for nodes, leaves in trees:
            kept = prune(nodes, leaves, k)
            depth_len = {}
            for n in kept:
                p, L = nodes[n]
                depth_len[n] = L + (depth_len[p] if p >= 0 else 0)
                tot += depth_len[n]
        return tot

    kmax = max(len(lv) for _n, lv in trees)
    K = 0
    for k in range(1, kmax + 1):
        if nu_for(k) <= budget:
            K = k
        else:
            break
    if K == 0:
        raise ValueError("c5: no K meets the token budget")
    parent, seg = [], []
    for nodes, leaves in trees:
        kept = prune(nodes, leaves, K)
        remap = {}
        for n in kept:
            p, L = nodes[n]
            remap[n] = len(seg)
            parent.append(remap[p] if p >= 0 else -1)
            seg.append(L)
    samples = list(range(len(seg)))
    return parent, seg, [blocks_exact(L) for L in seg], samples, K


_STRUCT = {"c1": _struct_c1, "c2": _struct_c2, "c2-small": _struct_c2_small, "c3": _struct_c3, "c4": _struct_c4}


def tree_stats(tree: Tree, hq: int, d: int) -> dict:
    """Workload accounting: shared/unshared token counts, visible (q,k) pairs, FLOPs."""
    off = tree.node_offsets()
    L = tree.seg_len.astype(np.int64)
    ns = int(L.sum())
    refc = sample_refcounts(tree)
    path_len = off + L
    nu = int(sum(int(path_len[e]) for e in tree.sample_end))
    nvis = int(np.sum(L * off + L * (L + 1) // 2))
    shared_tokens = int(np.sum(L * refc * (refc >= 2)))
    return {
        "nodes": tree.num_nodes,
        "samples": int(tree.sample_end.shape[0]),
        "blocks": int(tree.blk_cap.shape[0]),
        "pool_slots": tree.pool_slots,
        "Ns": ns,
        "Nu": nu,
        "redundancy": 1.0 - ns / nu,
        "pmr": shared_tokens / nu,
        "max_sample": int(max(int(path_len[e]) for e in tree.sample_end)),
        "sum_nvis": nvis,
        "flop_fwd": 4 * d * hq * nvis,
        "flop_bwd": 10 * d * hq * nvis,
        "flop_alg": 14 * d * hq * nvis,
        "min_seg": int(L.min()),
        "max_seg": int(L.max()),
    }


def sample_refcounts(tree: Tree) -> np.ndarray:
    """Number of samples whose root-to-endpoint path contains each node."""
    rc = np.zeros(tree.num_nodes, dtype=np.int64)
    for e in tree.sample_end:
        for n in tree.path(int(e)):
            rc[n] += 1
    return rc


# --------------------------------------------------------------------------- public API

def make_tree(name: str) -> Tuple[Tree, dict]:
    """Tree structure of a named config (pool bases in identity order; no tensor draws)."""
    seed = CONFIGS[name][0]
    rng_tree, _ = [np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(2)]
    extra = {}
    if name == "c5":
        parent, seg, blocks, samples, K = _struct_c5(rng_tree)
        extra["K"] = K
    else:
        parent, seg, blocks, samples = _STRUCT[name](rng_tree)
    return _make_tree(parent, seg, blocks, samples), extra


def make(name: str, tensors: bool = True) -> Workload:
    """Full workload: tree, page pool (permuted block order) and input tensors."""
    seed, hq, hkv, d, dtype, sigma, _desc = CONFIGS[name]
    rng_tree, rng_tensor = [np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(2)]
    if name == "c5":
        parent, seg, blocks, samples, _K = _struct_c5(rng_tree)
    else:
        parent, seg, blocks, samples = _STRUCT[name](rng_tree)
    ns = int(np.sum(seg))
    wl = Workload(name=name, tree=None, hq=hq, hkv=hkv, d=d, dtype=dtype, scale=1.0 / math.sqrt(d))
    if tensors:
        wl.Q = _draw(rng_tensor, (ns, hq, d), sigma, dtype)
        wl.K = _draw(rng_tensor, (ns, hkv, d), sigma, dtype)
        wl.V = _draw(rng_tensor, (ns, hkv, d), sigma, dtype)
        wl.dO = _draw(rng_tensor, (ns, hq, d), 1.0, dtype)
    else:
        _skip_draw(rng_tensor, ns * hq * d * 2 + ns * hkv * d * 2)
    nb = sum(len(b) for b in blocks)
    perm = rng_tensor.permutation(nb)
    wl.tree = _make_tree(parent, seg, blocks, samples, perm=perm)
    if tensors:
        wl.K_pool, wl.V_pool = scatter_pool(wl.tree, wl.K, wl.V)
    return wl


def add_attention_sink(wl: Workload, key_rows: Sequence[int], logit: float) -> Workload:
    """Attention-sink inputs: add to every query of every head h a multiple of the key of each
    row in ``key_rows`` (kv head h // G), so that scale * q . k of that key grows by ``logit``
    (about log(visible keys) puts half of a row's softmax weight on it).  Q is rounded to the
    workload dtype again; K, V and dO are unchanged.  Only the inputs change.
    """
    G = wl.hq // wl.hkv
    Q = wl.Q.astype(np.float64)
    for j in key_rows:
        for h in range(wl.hq):
            k = wl.K[int(j), h // G].astype(np.float64)
            Q[:, h] += (logit / wl.scale) * k / float(k @ k)
    wl.Q = _round(Q, wl.dtype)
    return wl


def call_subset(wl: Workload, ends: Sequence[int], external: Sequence[int] = ()) -> Tuple[Workload, np.ndarray]:
    """One call of a forest processed over several calls (micro-batches that reuse a cached prefix,
    Sec. 4.1.1 inter-batch sharing and 4.1.2 self-sequence sharing).

    The call's samples end at the forest nodes ``ends`` (a chunk of a long sequence ends at the
    chunk's node); it holds the nodes on their paths, in the forest's node order.  Forest nodes in ``external`` are cached by an earlier call: their K/V stay in the
    shared pool, they get no query rows (row_off = -1), and the backward adds this call's share of
    their dK/dV to what the earlier calls left.  Returns the call's workload (same pool, K/V and
    page blocks; Q and dO of its own rows; sample ends remapped) and, for each of its rows, the
    forest row it is.  The adjoint dO of a row is the forest's total adjoint of that token.
    """
    t = wl.tree
    ext = set(int(x) for x in external)
    keep = set()
    for e in ends:
        n = int(e)
        while n >= 0:
            keep.add(n)
            n = int(t.parent[n])
    nodes = sorted(keep)
    new_of = {n: i for i, n in enumerate(nodes)}
    parent = np.array([new_of[int(t.parent[n])] if t.parent[n] >= 0 else -1 for n in nodes], dtype=np.int32)
    seg = t.seg_len[nodes].astype(np.int32)
    row_off = np.full(len(nodes), -1, dtype=np.int64)
    rows = []
    cur = 0
    for i, n in enumerate(nodes):
        if n in ext:
            continue
        row_off[i] = cur
        rows.extend(range(int(t.row_off[n]), int(t.row_off[n]) + int(t.seg_len[n])))
        cur += int(t.seg_len[n])
    blk_ptr = [0]
    bidx = []
    for n in nodes:
        bidx.extend(range(int(t.blk_ptr[n]), int(t.blk_ptr[n + 1])))
        blk_ptr.append(len(bidx))
    bidx = np.asarray(bidx, dtype=np.int64)
    tree = Tree(parent=parent, seg_len=seg, row_off=row_off, blk_ptr=np.asarray(blk_ptr, dtype=np.int32),
                blk_base=t.blk_base[bidx], blk_cap=t.blk_cap[bidx], blk_len=t.blk_len[bidx], blk_pos=t.blk_pos[bidx],
                pool_slots=t.pool_slots,
                sample_end=np.array([new_of[int(e)] for e in ends], dtype=np.int32))
    rows = np.asarray(rows, dtype=np.int64)
    sub = Workload(name=f"{wl.name}-call", tree=tree, hq=wl.hq, hkv=wl.hkv, d=wl.d, dtype=wl.dtype, scale=wl.scale)
    if wl.Q is not None:
        sub.Q, sub.dO = wl.Q[rows], wl.dO[rows]
        sub.K, sub.V = wl.K[rows], wl.V[rows]
        sub.K_pool, sub.V_pool = wl.K_pool, wl.V_pool
    return sub, rows


def scatter_pool(tree: Tree, K: np.ndarray, V: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Place node-packed K/V rows into the page pool; pad slots get the sentinel."""
    hkv, d = K.shape[1], K.shape[2]
    kp = np.full((tree.pool_slots, hkv, d), SENTINEL, dtype=np.float32)
    vp = np.full((tree.pool_slots, hkv, d), SENTINEL, dtype=np.float32)
    slots = tree.row_slots()
    kp[slots] = K
    vp[slots] = V
    return kp, vp


def random_forest(seed: int, max_nodes: int = 12, max_seg: int = 40, hq: int = 4, hkv: int = 2,
                  d: int = 128, dtype: str = "bf16", sigma: float = 0.5, block_sizes=(1, 3, 16, 64),
                  min_seg: int = 1, shuffle_rows: bool = False, shuffle_pool: bool = True,
                  max_children: int = 0, tensors: bool = True) -> Workload:
    """Small random forest for exhaustive tests: random parents, lengths, block sizes and samples.

    Every node lies on at least one sample path.  ``shuffle_rows`` permutes the
    packed-row order of nodes (row_off stays a tiling of [0, Ns)).
    """
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, max_nodes + 1))
    parent = [-1]
    for i in range(1, n):
        if rng.random() < 0.15:
            parent.append(-1)
        else:
            cand = list(range(i))
            if max_children:
                kids = np.bincount([p for p in parent if p >= 0], minlength=i)
                cand = [c for c in cand if kids[c] < max_children] or [-1]
            parent.append(int(rng.choice(cand)) if cand != [-1] else -1)
    seg = [int(rng.integers(min_seg, max_seg + 1)) for _ in range(n)]
    blocks = []
    for L in seg:
        mode = int(rng.integers(0, 3))
        if mode == 0:
            blocks.append(blocks_exact(L))
        elif mode == 1:
            blocks.append(blocks_fixed(L, int(rng.choice(block_sizes))))
        else:
            # random partition with random spare capacity
            out, left = [], L
            while left > 0:
                ln = int(rng.integers(1, left + 1))
                out.append((ln + int(rng.integers(0, 3)), ln))
                left -= ln
            blocks.append(out)
    children = [[] for _ in range(n)]
    for i, p in enumerate(parent):
        if p >= 0:
            children[p].append(i)
    leaves = [i for i in range(n) if not children[i]]
    samples = set(leaves)
    for i in range(n):
        if rng.random() < 0.3:
            samples.add(i)
    samples = sorted(samples)
    rng.shuffle(samples)
    nb = sum(len(b) for b in blocks)
    perm = rng.permutation(nb) if shuffle_pool else None
    tree = _make_tree(parent, seg, blocks, samples, perm=perm)
    if shuffle_rows:
        order = rng.permutation(n)
        row_off = np.zeros(n, dtype=np.int64)
        cur = 0
        for i in order:
            row_off[i] = cur
            cur += seg[i]
        tree.row_off = row_off
    wl = Workload(name=f"rand{seed}", tree=tree, hq=hq, hkv=hkv, d=d, dtype=dtype,
                  scale=1.0 / math.sqrt(d))
    if tensors:
        ns = tree.num_rows
        wl.Q = _draw(rng, (ns, hq, d), sigma, dtype)
        wl.K = _draw(rng, (ns, hkv, d), sigma, dtype)
        wl.V = _draw(rng, (ns, hkv, d), sigma, dtype)
        wl.dO = _draw(rng, (ns, hq, d), 1.0, dtype)
        wl.K_pool, wl.V_pool = scatter_pool(tree, wl.K, wl.V)
    return wl


def custom(parent, seg_len, samples, hq=4, hkv=2, d=128, dtype="bf16", seed=0, sigma=0.5,
           block_policy=None, shuffle_pool=True, tensors=True) -> Workload:
    """A workload on a given tree shape (e.g. scaled-down versions of the named configs)."""
    rng = np.random.default_rng(seed)
    if block_policy is None:
        block_policy = lambda L: blocks_fixed(L, 64)
    blocks = [block_policy(L) for L in seg_len]
    nb = sum(len(b) for b in blocks)
    ns = int(np.sum(seg_len))
    wl = Workload(name="custom", tree=None, hq=hq, hkv=hkv, d=d, dtype=dtype, scale=1.0 / math.sqrt(d))
    if tensors:
        wl.Q = _draw(rng, (ns, hq, d), sigma, dtype)
        wl.K = _draw(rng, (ns, hkv, d), sigma, dtype)
        wl.V = _draw(rng, (ns, hkv, d), sigma, dtype)
        wl.dO = _draw(rng, (ns, hq, d), 1.0, dtype)
    perm = rng.permutation(nb) if shuffle_pool else None
    wl.tree = _make_tree(parent, seg_len, blocks, samples, perm=perm)
    if tensors:
        wl.K_pool, wl.V_pool = scatter_pool(wl.tree, wl.K, wl.V)
    return wl
