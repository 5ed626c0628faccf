"""Python binding of libpsattn (ctypes).  Argument marshalling only.

Every step of the forward and backward pass runs in the HIP kernels of
libpsattn.so; torch provides device memory and the current stream.  There
is no fallback: if the library is missing, or a tensor is not on a GPU,
the call raises.

Names follow the C ABI in include/psattn.h:
    Tree(...)                       psattn_tree_create / _upload / _destroy
    psattn_fwd(tree, Q, K, V)       -> (O, LSE)   (O_lo=: the bf16 rounding residual of O)
    psattn_bwd(tree, Q, K, V, O, LSE, dO) -> (dQ, dK, dV)   (O_lo=: Delta from O + O_lo)
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpsattn.so")

PSATTN_BF16 = 0
PSATTN_FP32 = 1
NOALLOC_SCRATCH_MIB = 128   # PSATTN_NOALLOC_SCRATCH_MIB: workspace limit of psattn_bwd_noalloc

STATUS = {
    0: "PSATTN_OK", -1: "PSATTN_E_INVALID_ARG", -2: "PSATTN_E_INVALID_TREE", -3: "PSATTN_E_BLOCK_RANGE",
    -4: "PSATTN_E_BLOCK_OVERLAP", -5: "PSATTN_E_BLOCK_COVERAGE", -6: "PSATTN_E_UNSUPPORTED",
    -7: "PSATTN_E_WORKSPACE", -8: "PSATTN_E_ALIGNMENT", -9: "PSATTN_E_HIP", -10: "PSATTN_E_NOT_UPLOADED",
    -11: "PSATTN_E_INTERNAL",
}

EXPORTED = [
    "psattn_tree_create", "psattn_tree_destroy", "psattn_tree_device_bytes", "psattn_tree_upload",
    "psattn_workspace_size", "psattn_fwd", "psattn_bwd", "psattn_bwd_noalloc", "psattn_tree_refcounts",
    "psattn_tree_get_info",
    "psattn_tree_plan_array", "psattn_profile_enable", "psattn_profile_reset", "psattn_profile_read",
    "psattn_status_string", "psattn_last_error",
    "psattn_kvm_plan", "psattn_kvm_destroy", "psattn_kvm_call_desc", "psattn_kvm_events", "psattn_kvm_get_stats",
    "psattn_sched_fit", "psattn_sched_group_costs", "psattn_sched_place", "psattn_sched_microbatch",
    "psattn_sched_mb_get", "psattn_sched_mb_destroy", "psattn_rope", "psattn_kv_scatter", "psattn_kv_gather",
]

KVM_EVENTS = {0: "alloc", 1: "refill", 2: "evict", 3: "free"}

PLAN_ARRAYS = {"row_pos": 0, "q_list": 1, "kv_list": 2, "fwd_items": 3, "fwd_merges": 4, "bkv_items": 5,
               "bkv_reduces": 6, "pad_slots": 7, "row_slot": 8, "q_pos": 9}


class PsattnError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status
        self.name = STATUS.get(status, str(status))


class Block(ctypes.Structure):
    _fields_ = [("base", ctypes.c_int64), ("capacity", ctypes.c_int32), ("len", ctypes.c_int32),
                ("pos", ctypes.c_int32), ("refcount", ctypes.c_int32)]


_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)


class TreeDesc(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int32), ("parent", _i32p), ("seg_len", _i32p), ("row_off", _i64p),
                ("blk_ptr", _i32p), ("blocks", ctypes.POINTER(Block)), ("pool_slots", ctypes.c_int64),
                ("num_samples", ctypes.c_int32), ("sample_end", _i32p), ("hq", ctypes.c_int32),
                ("hkv", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("softmax_scale", ctypes.c_float),
                ("dtype", ctypes.c_int32)]


class KvmEvent(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("node", ctypes.c_int32), ("num_blocks", ctypes.c_int32),
                ("capacity", ctypes.c_int32), ("base", ctypes.c_int64)]


class KvmOpts(ctypes.Structure):
    _fields_ = [("capacity_slots", ctypes.c_int64), ("block_size", ctypes.c_int32), ("dbc", ctypes.c_int32),
                ("reserved", ctypes.c_int32 * 4)]


class KvmStats(ctypes.Structure):
    _fields_ = [("peak_slots", ctypes.c_int64), ("final_slots", ctypes.c_int64), ("evictions", ctypes.c_int64),
                ("refilled_tokens", ctypes.c_int64), ("allocated_tokens", ctypes.c_int64),
                ("num_calls", ctypes.c_int32), ("pad_", ctypes.c_int32)]


_f64p = ctypes.POINTER(ctypes.c_double)


class SchedMbView(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_int32), ("parent", _i32p), ("seg_len", _i32p), ("src_node", _i32p),
                ("src_offset", _i32p), ("num_chunks", ctypes.c_int32), ("chunk_end", _i32p),
                ("chunk_micro_batch", _i32p), ("chunk_sample", _i32p), ("num_micro_batches", ctypes.c_int32),
                ("micro_batch_cost", _f64p)]


class PlanOpts(ctypes.Structure):
    _fields_ = [("fwd_kv_split", ctypes.c_int32), ("bwd_q_chunk", ctypes.c_int32), ("num_cus", ctypes.c_int32),
                ("reserved", ctypes.c_int32 * 5)]


class TreeInfo(ctypes.Structure):
    _fields_ = [("num_rows", ctypes.c_int64), ("unshared_tokens", ctypes.c_int64), ("visible_pairs", ctypes.c_int64),
                ("fwd_items", ctypes.c_int64), ("fwd_merges", ctypes.c_int64), ("bkv_items", ctypes.c_int64),
                ("bkv_reduces", ctypes.c_int64), ("pad_slots", ctypes.c_int64), ("fwd_partial_rows", ctypes.c_int64),
                ("bkv_partial_tiles", ctypes.c_int64), ("plan_bytes", ctypes.c_int64), ("q_tile_rows", ctypes.c_int32),
                ("kv_tile_keys", ctypes.c_int32), ("bkv_tile_keys", ctypes.c_int32), ("head_chunk", ctypes.c_int32)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


_LIB = None


def lib() -> ctypes.CDLL:
    """Load libpsattn.so (built in-tree by __graft_entry__.build()); raise if it is missing."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        vp, sz = ctypes.c_void_p, ctypes.c_size_t
        L.psattn_tree_create.argtypes = [ctypes.POINTER(TreeDesc), ctypes.POINTER(PlanOpts), ctypes.POINTER(vp)]
        L.psattn_tree_destroy.argtypes = [vp]
        L.psattn_tree_destroy.restype = None
        L.psattn_tree_device_bytes.argtypes = [vp, ctypes.POINTER(sz)]
        L.psattn_tree_upload.argtypes = [vp, vp, sz, vp]
        L.psattn_workspace_size.argtypes = [vp, ctypes.c_int, ctypes.POINTER(sz)]
        L.psattn_fwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.psattn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.psattn_bwd_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.psattn_tree_refcounts.argtypes = [vp, _i32p]
        L.psattn_tree_get_info.argtypes = [vp, ctypes.POINTER(TreeInfo)]
        L.psattn_tree_plan_array.argtypes = [vp, ctypes.c_int, ctypes.POINTER(_i32p), _i64p, _i32p]
        L.psattn_profile_enable.argtypes = [ctypes.c_int]
        L.psattn_profile_reset.argtypes = []
        L.psattn_profile_read.argtypes = [ctypes.c_int32, _i32p, ctypes.POINTER(ctypes.c_char_p), _i64p,
                                          ctypes.POINTER(ctypes.c_double)]
        L.psattn_status_string.argtypes = [ctypes.c_int]
        L.psattn_status_string.restype = ctypes.c_char_p
        L.psattn_last_error.argtypes = []
        L.psattn_last_error.restype = ctypes.c_char_p
        L.psattn_kvm_plan.argtypes = [ctypes.c_int32, _i32p, _i32p, ctypes.c_int32, _i32p, _i32p,
                                      ctypes.POINTER(KvmOpts), ctypes.POINTER(vp)]
        L.psattn_kvm_destroy.argtypes = [vp]
        L.psattn_kvm_destroy.restype = None
        L.psattn_kvm_call_desc.argtypes = [vp, ctypes.c_int32, ctypes.POINTER(TreeDesc), ctypes.POINTER(_i32p)]
        L.psattn_kvm_events.argtypes = [vp, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.POINTER(KvmEvent)),
                                        _i32p]
        L.psattn_kvm_get_stats.argtypes = [vp, ctypes.POINTER(KvmStats), _i64p]
        L.psattn_sched_fit.argtypes = [ctypes.c_int32, _f64p, _f64p, _f64p, _f64p]
        L.psattn_sched_group_costs.argtypes = [ctypes.c_int32, _i32p, _i32p, ctypes.c_int32, _i32p, _i32p,
                                               ctypes.c_int32, _f64p, _f64p]
        L.psattn_sched_place.argtypes = [ctypes.c_int32, _f64p, ctypes.c_int32, _i32p, _f64p]
        L.psattn_sched_microbatch.argtypes = [ctypes.c_int32, _i32p, _i32p, ctypes.c_int32, _i32p, _f64p,
                                              ctypes.c_int32, ctypes.POINTER(vp)]
        L.psattn_sched_mb_get.argtypes = [vp, ctypes.POINTER(SchedMbView)]
        L.psattn_sched_mb_destroy.argtypes = [vp]
        L.psattn_rope.argtypes = [vp, vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_float, ctypes.c_int32, vp]
        L.psattn_kv_scatter.argtypes = [vp, vp, vp, vp, vp, vp]
        L.psattn_kv_gather.argtypes = [vp, vp, vp, vp, vp, vp]
        L.psattn_sched_mb_destroy.restype = None
        for name in EXPORTED:
            if name not in ("psattn_tree_destroy", "psattn_status_string", "psattn_last_error"):
                getattr(L, name).restype = ctypes.c_int
        _LIB = L
    return _LIB


def _check(status: int) -> None:
    if status != 0:
        raise PsattnError(status, lib().psattn_last_error().decode())


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


class Tree:
    """A validated prefix tree + page table + work plan (psattn_tree_create).

    Arrays follow psattn_tree_desc.  ``opts`` is a dict of psattn_plan_opts
    fields.  Call :meth:`upload` (or pass ``device``) before psattn_fwd/bwd.
    """

    def __init__(self, parent, seg_len, row_off, blk_ptr, blk_base, blk_cap, blk_len, blk_pos, pool_slots,
                 sample_end, hq, hkv, head_dim, softmax_scale, dtype="bf16", blk_refcount=None, opts=None,
                 device=None):
        L = lib()
        self._handle = None
        self.parent = np.ascontiguousarray(parent, dtype=np.int32)
        self.seg_len = np.ascontiguousarray(seg_len, dtype=np.int32)
        self.row_off = np.ascontiguousarray(row_off, dtype=np.int64)
        self.blk_ptr = np.ascontiguousarray(blk_ptr, dtype=np.int32)
        self.sample_end = np.ascontiguousarray(sample_end, dtype=np.int32)
        nb = len(blk_base)
        blocks = (Block * max(nb, 1))()
        rc = np.zeros(nb, dtype=np.int64) if blk_refcount is None else np.asarray(blk_refcount)
        for i in range(nb):
            blocks[i] = Block(int(blk_base[i]), int(blk_cap[i]), int(blk_len[i]), int(blk_pos[i]), int(rc[i]))
        self.dtype = dtype
        self.hq, self.hkv, self.head_dim = int(hq), int(hkv), int(head_dim)
        self.scale = float(softmax_scale)
        self.pool_slots = int(pool_slots)
        desc = TreeDesc(len(self.parent), _ptr(self.parent, ctypes.c_int32), _ptr(self.seg_len, ctypes.c_int32),
                        _ptr(self.row_off, ctypes.c_int64), _ptr(self.blk_ptr, ctypes.c_int32), blocks,
                        int(pool_slots), len(self.sample_end), _ptr(self.sample_end, ctypes.c_int32), self.hq,
                        self.hkv, self.head_dim, self.scale, PSATTN_BF16 if dtype == "bf16" else PSATTN_FP32)
        o = PlanOpts()
        for k, v in (opts or {}).items():
            if k == "reserved":
                for i, x in enumerate(v):
                    o.reserved[i] = int(x)
            else:
                setattr(o, k, int(v))
        h = ctypes.c_void_p()
        _check(L.psattn_tree_create(ctypes.byref(desc), ctypes.byref(o), ctypes.byref(h)))
        self._handle = h
        info = TreeInfo()
        _check(L.psattn_tree_get_info(h, ctypes.byref(info)))
        self.info = info.as_dict()
        self.num_rows = int(self.info["num_rows"])
        self._plan_buf = None
        self._ws = {}
        if device is not None:
            self.upload(device)

    @classmethod
    def from_workload(cls, wl, opts=None, device=None, **kw):
        t = wl.tree
        return cls(t.parent, t.seg_len, t.row_off, t.blk_ptr, t.blk_base, t.blk_cap, t.blk_len, t.blk_pos,
                   t.pool_slots, t.sample_end, wl.hq, wl.hkv, wl.d, wl.scale, dtype=wl.dtype, opts=opts,
                   device=device, **kw)

    @property
    def handle(self):
        return self._handle

    def __del__(self):
        if getattr(self, "_handle", None) is not None and _LIB is not None:
            _LIB.psattn_tree_destroy(self._handle)
            self._handle = None

    def device_bytes(self) -> int:
        n = ctypes.c_size_t()
        _check(lib().psattn_tree_device_bytes(self._handle, ctypes.byref(n)))
        return n.value

    def workspace_size(self, pass_: int) -> int:
        n = ctypes.c_size_t()
        _check(lib().psattn_workspace_size(self._handle, pass_, ctypes.byref(n)))
        return n.value

    def upload(self, device="cuda"):
        import torch
        nbytes = self.device_bytes()
        buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
        stream = torch.cuda.current_stream(buf.device).cuda_stream
        _check(lib().psattn_tree_upload(self._handle, ctypes.c_void_p(buf.data_ptr()), nbytes, ctypes.c_void_p(stream)))
        self._plan_buf = buf
        self.device = buf.device
        return self

    def workspace(self, pass_: int):
        """A cached workspace tensor for pass 0 (fwd) or 1 (bwd), allocated through torch."""
        import torch
        n = self.workspace_size(pass_)
        ws = self._ws.get(pass_)
        if ws is None or ws.numel() < n:
            ws = torch.empty(max(n, 256), dtype=torch.uint8, device=self.device)
            self._ws[pass_] = ws
        return ws

    def refcounts(self) -> np.ndarray:
        out = np.zeros(len(self.parent), dtype=np.int32)
        _check(lib().psattn_tree_refcounts(self._handle, _ptr(out, ctypes.c_int32)))
        return out

    def plan_array(self, name: str) -> np.ndarray:
        data = _i32p()
        count = ctypes.c_int64()
        width = ctypes.c_int32()
        _check(lib().psattn_tree_plan_array(self._handle, PLAN_ARRAYS[name], ctypes.byref(data), ctypes.byref(count),
                                            ctypes.byref(width)))
        n = count.value * width.value
        if n == 0:
            return np.zeros((0, width.value) if width.value > 1 else (0,), dtype=np.int32)
        arr = np.ctypeslib.as_array(data, shape=(n,)).copy()
        return arr.reshape(count.value, width.value) if width.value > 1 else arr


def _torch_dtype(tree):
    import torch
    return torch.bfloat16 if tree.dtype == "bf16" else torch.float32


def _need(t, shape, dtype, name):
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise RuntimeError(f"{name} must be on a GPU (the HIP path has no CPU fallback)")
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype or not t.is_contiguous():
        raise ValueError(f"{name}: expected contiguous {dtype} {tuple(shape)}, got {t.dtype} {tuple(t.shape)}")


def _vp(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def psattn_fwd(tree: Tree, Q, K, V, O=None, LSE=None, ws=None, O_lo=None):
    """Forward pass on the current stream; returns (O [Ns,Hq,d], LSE [Hq,Ns] fp32).  O_lo (bf16
    trees, optional, like O): filled with the rounding residual of O, for psattn_bwd."""
    import torch
    if tree._plan_buf is None:
        raise RuntimeError("tree not uploaded (call Tree.upload)")
    dt = _torch_dtype(tree)
    ns, hq, hkv, d = tree.num_rows, tree.hq, tree.hkv, tree.head_dim
    _need(Q, (ns, hq, d), dt, "Q")
    _need(K, (tree.pool_slots, hkv, d), dt, "K")
    _need(V, (tree.pool_slots, hkv, d), dt, "V")
    if O is None:
        O = torch.empty((ns, hq, d), dtype=dt, device=Q.device)
    if LSE is None:
        LSE = torch.empty((hq, ns), dtype=torch.float32, device=Q.device)
    _need(O, (ns, hq, d), dt, "O")
    _need(LSE, (hq, ns), torch.float32, "LSE")
    if O_lo is not None:
        _need(O_lo, (ns, hq, d), dt, "O_lo")
    if ws is None:
        ws = tree.workspace(0)
    stream = torch.cuda.current_stream(Q.device).cuda_stream
    _check(lib().psattn_fwd(tree.handle, _vp(Q), _vp(K), _vp(V), _vp(O), _vp(LSE), _vp(O_lo), _vp(ws), ws.numel(),
                            ctypes.c_void_p(stream)))
    return O, LSE


def psattn_bwd(tree: Tree, Q, K, V, O, LSE, dO, dQ=None, dK=None, dV=None, ws=None, O_lo=None):
    """Backward pass on the current stream; returns (dQ, dK, dV), all fp32.  O_lo: the forward's
    residual of O, if it was produced (Delta then comes from O + O_lo)."""
    import torch
    if tree._plan_buf is None:
        raise RuntimeError("tree not uploaded (call Tree.upload)")
    dt = _torch_dtype(tree)
    ns, hq, hkv, d, ps = tree.num_rows, tree.hq, tree.hkv, tree.head_dim, tree.pool_slots
    _need(Q, (ns, hq, d), dt, "Q")
    _need(K, (ps, hkv, d), dt, "K")
    _need(V, (ps, hkv, d), dt, "V")
    _need(O, (ns, hq, d), dt, "O")
    _need(LSE, (hq, ns), torch.float32, "LSE")
    _need(dO, (ns, hq, d), dt, "dO")
    if O_lo is not None:
        _need(O_lo, (ns, hq, d), dt, "O_lo")
    f32 = torch.float32
    if dQ is None:
        dQ = torch.empty((ns, hq, d), dtype=f32, device=Q.device)
    if dK is None:
        dK = torch.empty((ps, hkv, d), dtype=f32, device=Q.device)
    if dV is None:
        dV = torch.empty((ps, hkv, d), dtype=f32, device=Q.device)
    _need(dQ, (ns, hq, d), f32, "dQ")
    _need(dK, (ps, hkv, d), f32, "dK")
    _need(dV, (ps, hkv, d), f32, "dV")
    if ws is None:
        ws = tree.workspace(1)
    stream = torch.cuda.current_stream(Q.device).cuda_stream
    _check(lib().psattn_bwd(tree.handle, _vp(Q), _vp(K), _vp(V), _vp(O), _vp(LSE), _vp(O_lo), _vp(dO), _vp(dQ),
                            _vp(dK), _vp(dV), _vp(ws), ws.numel(), ctypes.c_void_p(stream)))
    return dQ, dK, dV


def psattn_bwd_noalloc(tree: Tree, Q, K, V, O, LSE, dO, dQ, dK, dV, O_lo=None):
    """psattn_bwd with its workspace in the library's per-GPU device array (no workspace argument,
    nothing allocated by the library); the output tensors are the caller's."""
    import torch
    if tree._plan_buf is None:
        raise RuntimeError("tree not uploaded (call Tree.upload)")
    dt = _torch_dtype(tree)
    ns, hq, hkv, d, ps = tree.num_rows, tree.hq, tree.hkv, tree.head_dim, tree.pool_slots
    f32 = torch.float32
    for x, shape, t, name in ((Q, (ns, hq, d), dt, "Q"), (K, (ps, hkv, d), dt, "K"), (V, (ps, hkv, d), dt, "V"),
                              (O, (ns, hq, d), dt, "O"), (LSE, (hq, ns), f32, "LSE"), (dO, (ns, hq, d), dt, "dO"),
                              (dQ, (ns, hq, d), f32, "dQ"), (dK, (ps, hkv, d), f32, "dK"), (dV, (ps, hkv, d), f32, "dV")):
        _need(x, shape, t, name)
    if O_lo is not None:
        _need(O_lo, (ns, hq, d), dt, "O_lo")
    stream = torch.cuda.current_stream(Q.device).cuda_stream
    _check(lib().psattn_bwd_noalloc(tree.handle, _vp(Q), _vp(K), _vp(V), _vp(O), _vp(LSE), _vp(O_lo), _vp(dO),
                                    _vp(dQ), _vp(dK), _vp(dV), ctypes.c_void_p(stream)))
    return dQ, dK, dV


class KVCachePlan:
    """The adaptive KV cache manager's plan of a schedule (psattn_kvm_plan): a forest, the call
    (micro-batch) of each sample, and a pool of ``capacity`` slots."""

    def __init__(self, parent, seg_len, sample_end, call_of_sample, capacity, block_size=0, dbc=True):
        L = lib()
        self._handle = None
        self.parent = np.ascontiguousarray(parent, dtype=np.int32)
        self.seg_len = np.ascontiguousarray(seg_len, dtype=np.int32)
        self.sample_end = np.ascontiguousarray(sample_end, dtype=np.int32)
        self.call_of_sample = np.ascontiguousarray(call_of_sample, dtype=np.int32)
        o = KvmOpts(int(capacity), int(block_size), 1 if dbc else 0)
        h = ctypes.c_void_p()
        _check(L.psattn_kvm_plan(len(self.parent), _ptr(self.parent, ctypes.c_int32), _ptr(self.seg_len, ctypes.c_int32),
                                 len(self.sample_end), _ptr(self.sample_end, ctypes.c_int32),
                                 _ptr(self.call_of_sample, ctypes.c_int32), ctypes.byref(o), ctypes.byref(h)))
        self._handle = h
        st = KvmStats()
        _check(L.psattn_kvm_get_stats(h, ctypes.byref(st), None))
        self.num_calls = st.num_calls
        used = np.zeros(max(self.num_calls, 1), dtype=np.int64)
        _check(L.psattn_kvm_get_stats(h, ctypes.byref(st), _ptr(used, ctypes.c_int64)))
        self.stats = {k: getattr(st, k) for k, _ in KvmStats._fields_ if k != "pad_"}
        self.used_per_call = used[:self.num_calls]

    def __del__(self):
        if getattr(self, "_handle", None) is not None:
            lib().psattn_kvm_destroy(self._handle)
            self._handle = None

    def call(self, c: int) -> dict:
        """Call c's descriptor arrays (numpy copies) and its forest node ids."""
        d = TreeDesc()
        ids = _i32p()
        _check(lib().psattn_kvm_call_desc(self._handle, int(c), ctypes.byref(d), ctypes.byref(ids)))
        n = d.num_nodes
        nb = d.blk_ptr[n]
        arr = lambda p, k: np.ctypeslib.as_array(p, shape=(k,)).copy() if k else np.zeros(0, dtype=np.int32)
        blocks = [d.blocks[i] for i in range(nb)]
        return {"node_ids": arr(ids, n), "parent": arr(d.parent, n), "seg_len": arr(d.seg_len, n),
                "row_off": arr(d.row_off, n), "blk_ptr": arr(d.blk_ptr, n + 1),
                "blk_base": np.array([b.base for b in blocks], dtype=np.int64),
                "blk_cap": np.array([b.capacity for b in blocks], dtype=np.int32),
                "blk_len": np.array([b.len for b in blocks], dtype=np.int32),
                "blk_pos": np.array([b.pos for b in blocks], dtype=np.int32), "pool_slots": int(d.pool_slots),
                "sample_end": arr(d.sample_end, d.num_samples)}

    def events(self, c: int, phase: int) -> list:
        """[(kind, forest node, num_blocks, capacity, base)] before (phase 0) or after (1) call c."""
        ev = ctypes.POINTER(KvmEvent)()
        n = ctypes.c_int32()
        _check(lib().psattn_kvm_events(self._handle, int(c), int(phase), ctypes.byref(ev), ctypes.byref(n)))
        return [(KVM_EVENTS[ev[i].kind], ev[i].node, ev[i].num_blocks, ev[i].capacity, ev[i].base) for i in range(n.value)]


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def sched_fit(l_suf, l, t) -> np.ndarray:
    """(a1, a2, a3) of Eq. "single_sequence" fitted to measured runs (psattn_sched_fit)."""
    l_suf, l, t = _f64(l_suf), _f64(l), _f64(t)
    alpha = np.zeros(3)
    _check(lib().psattn_sched_fit(len(t), _ptr(l_suf, ctypes.c_double), _ptr(l, ctypes.c_double),
                                  _ptr(t, ctypes.c_double), _ptr(alpha, ctypes.c_double)))
    return alpha


def sched_group_costs(parent, seg_len, sample_end, group_of_sample, num_groups, alpha) -> np.ndarray:
    parent, seg_len, sample_end, gos, alpha = _i32(parent), _i32(seg_len), _i32(sample_end), _i32(group_of_sample), _f64(alpha)
    out = np.zeros(int(num_groups))
    _check(lib().psattn_sched_group_costs(len(parent), _ptr(parent, ctypes.c_int32), _ptr(seg_len, ctypes.c_int32),
                                          len(sample_end), _ptr(sample_end, ctypes.c_int32), _ptr(gos, ctypes.c_int32),
                                          int(num_groups), _ptr(alpha, ctypes.c_double), _ptr(out, ctypes.c_double)))
    return out


def sched_place(group_cost, num_workers):
    """(worker of each group, load of each worker) of the greedy placement (psattn_sched_place)."""
    c = _f64(group_cost)
    w = np.zeros(len(c), dtype=np.int32)
    load = np.zeros(int(num_workers))
    _check(lib().psattn_sched_place(len(c), _ptr(c, ctypes.c_double), int(num_workers), _ptr(w, ctypes.c_int32),
                                    _ptr(load, ctypes.c_double)))
    return w, load


def sched_microbatch(parent, seg_len, sample_end, alpha, num_micro_batches) -> dict:
    """Token-wise micro-batching (psattn_sched_microbatch): the refined forest and its chunks."""
    parent, seg_len, sample_end, alpha = _i32(parent), _i32(seg_len), _i32(sample_end), _f64(alpha)
    h = ctypes.c_void_p()
    L = lib()
    _check(L.psattn_sched_microbatch(len(parent), _ptr(parent, ctypes.c_int32), _ptr(seg_len, ctypes.c_int32),
                                     len(sample_end), _ptr(sample_end, ctypes.c_int32), _ptr(alpha, ctypes.c_double),
                                     int(num_micro_batches), ctypes.byref(h)))
    try:
        v = SchedMbView()
        _check(L.psattn_sched_mb_get(h, ctypes.byref(v)))
        arr = lambda p, k, dt=np.int32: np.ctypeslib.as_array(p, shape=(k,)).astype(dt) if k else np.zeros(0, dt)
        return {"parent": arr(v.parent, v.num_nodes), "seg_len": arr(v.seg_len, v.num_nodes),
                "src_node": arr(v.src_node, v.num_nodes), "src_offset": arr(v.src_offset, v.num_nodes),
                "chunk_end": arr(v.chunk_end, v.num_chunks), "chunk_micro_batch": arr(v.chunk_micro_batch, v.num_chunks),
                "chunk_sample": arr(v.chunk_sample, v.num_chunks),
                "micro_batch_cost": arr(v.micro_batch_cost, v.num_micro_batches, np.float64)}
    finally:
        L.psattn_sched_mb_destroy(h)


def psattn_rope(tree: Tree, X, theta: float = 10000.0, inverse: bool = False):
    """Rotary embedding of X [Ns][heads][d] (bf16 or fp32) in place by each row's sequence position."""
    import torch
    if X.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("X must be bf16 or fp32")
    _need(X, (tree.num_rows, X.shape[1], tree.head_dim), X.dtype, "X")
    dt = PSATTN_BF16 if X.dtype == torch.bfloat16 else PSATTN_FP32
    _check(lib().psattn_rope(tree.handle, _vp(X), dt, int(X.shape[1]), float(theta), 1 if inverse else 0,
                             ctypes.c_void_p(torch.cuda.current_stream(X.device).cuda_stream)))
    return X


def psattn_kv_scatter(tree: Tree, K_rows, V_rows, K, V):
    """K/V rows [Ns][Hkv][d] written into their pool slots of K, V."""
    import torch
    dt = _torch_dtype(tree)
    for x, shape, name in ((K_rows, (tree.num_rows, tree.hkv, tree.head_dim), "K_rows"),
                           (V_rows, (tree.num_rows, tree.hkv, tree.head_dim), "V_rows"),
                           (K, (tree.pool_slots, tree.hkv, tree.head_dim), "K"),
                           (V, (tree.pool_slots, tree.hkv, tree.head_dim), "V")):
        _need(x, shape, dt, name)
    _check(lib().psattn_kv_scatter(tree.handle, _vp(K_rows), _vp(V_rows), _vp(K), _vp(V),
                                   ctypes.c_void_p(torch.cuda.current_stream(K.device).cuda_stream)))


def psattn_kv_gather(tree: Tree, dK, dV, dK_rows=None, dV_rows=None):
    """dK/dV of each row's pool slot -> rows [Ns][Hkv][d] (fp32)."""
    import torch
    shape = (tree.num_rows, tree.hkv, tree.head_dim)
    dK_rows = torch.empty(shape, dtype=torch.float32, device=dK.device) if dK_rows is None else dK_rows
    dV_rows = torch.empty(shape, dtype=torch.float32, device=dK.device) if dV_rows is None else dV_rows
    for x, shp, name in ((dK, (tree.pool_slots,) + shape[1:], "dK"), (dV, (tree.pool_slots,) + shape[1:], "dV"),
                         (dK_rows, shape, "dK_rows"), (dV_rows, shape, "dV_rows")):
        _need(x, shp, torch.float32, name)
    _check(lib().psattn_kv_gather(tree.handle, _vp(dK), _vp(dV), _vp(dK_rows), _vp(dV_rows),
                                  ctypes.c_void_p(torch.cuda.current_stream(dK.device).cuda_stream)))
    return dK_rows, dV_rows


def psattn_profile_enable(on: bool = True) -> None:
    _check(lib().psattn_profile_enable(1 if on else 0))


def psattn_profile_reset() -> None:
    _check(lib().psattn_profile_reset())


def psattn_profile_read() -> dict:
    """{kernel name: (launches, total ms)} since the last reset (waits for the recorded events)."""
    n = ctypes.c_int32()
    cap = 16
    names = (ctypes.c_char_p * cap)()
    launches = (ctypes.c_int64 * cap)()
    ms = (ctypes.c_double * cap)()
    _check(lib().psattn_profile_read(cap, ctypes.byref(n), names, launches, ms))
    return {names[i].decode(): (int(launches[i]), float(ms[i])) for i in range(min(n.value, cap))}
