"""Thin ctypes binding of libtangram_hip.so (include/tangram.h).

Argument marshalling only: every step of the plan search runs in the HIP
kernels of the library.  Device buffers are torch tensors on the GPU; the
stream passed to the library is torch's current HIP stream.  There is no CPU
fallback: importing this module without the built library raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtangram_hip.so")

TG_OK, TG_EINVAL, TG_ENOMEM, TG_EDEVICE, TG_ECAPACITY, TG_ENOPLAN = 0, -1, -2, -3, -4, -5
LAYER_FIELDS = ("fwd_flops", "dense_params", "expert_params", "act_stash_bytes",
                "tp_comm_bytes", "a2a_bytes", "out_act_bytes", "cp_comm_bytes")


class TgLayer(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int64) for f in LAYER_FIELDS]


class TgIsland(ctypes.Structure):
    _fields_ = [("n_gpus", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("peak_flops", ctypes.c_double), ("hbm_bytes", ctypes.c_double),
                ("intra_bw", ctypes.c_double), ("host_bw", ctypes.c_double)]


class TgSpace(ctypes.Structure):
    _fields_ = [("global_batch", ctypes.c_int64), ("n_experts", ctypes.c_int32),
                ("n_tp", ctypes.c_int32), ("tp", ctypes.c_int32 * 8),
                ("n_ep", ctypes.c_int32), ("ep", ctypes.c_int32 * 8),
                ("n_mb", ctypes.c_int32), ("mb", ctypes.c_int32 * 8),
                ("zero_mask", ctypes.c_uint32), ("reserved", ctypes.c_int32),
                ("eta", ctypes.c_double), ("mem_frac", ctypes.c_double),
                ("n_cp", ctypes.c_int32), ("cp", ctypes.c_int32 * 8),
                ("recompute_mask", ctypes.c_uint32), ("offload_mask", ctypes.c_uint32),
                ("reserved2", ctypes.c_int32), ("imbalance_eps", ctypes.c_double)]


PAIR_FIELDS = ("i", "j", "island", "tp", "cp", "dp", "ep", "zero", "recompute", "offload", "mb")


class TgPair(ctypes.Structure):
    _fields_ = [(f, ctypes.c_int32) for f in PAIR_FIELDS + ("reserved",)]


class TgStage(ctypes.Structure):
    _fields_ = [("island", ctypes.c_int32), ("first_layer", ctypes.c_int32),
                ("end_layer", ctypes.c_int32), ("tp", ctypes.c_int32), ("cp", ctypes.c_int32),
                ("dp", ctypes.c_int32), ("ep", ctypes.c_int32), ("zero", ctypes.c_int32),
                ("recompute", ctypes.c_int32), ("offload", ctypes.c_int32), ("mb", ctypes.c_int32),
                ("depth", ctypes.c_int32),
                ("pair_index", ctypes.c_int64), ("cost", ctypes.c_double),
                ("mem_bytes", ctypes.c_double), ("link_out", ctypes.c_double)]


class TgPlan(ctypes.Structure):
    _fields_ = [("b", ctypes.c_int32), ("m", ctypes.c_int32), ("S", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("P", ctypes.c_double), ("F", ctypes.c_double),
                ("T", ctypes.c_double), ("stage", TgStage * 255)]


class TgInfo(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("K", ctypes.c_int32), ("n_b", ctypes.c_int32),
                ("dense", ctypes.c_int32), ("NS", ctypes.c_int64), ("n_configs", ctypes.c_int64),
                ("N", ctypes.c_int64), ("n_compatible_configs", ctypes.c_int64),
                ("n_slice_classes", ctypes.c_int64)]


class TangramError(RuntimeError):
    def __init__(self, status, what, msg):
        super().__init__(f"{what} failed with status {status}: {msg}")
        self.status = status


EXPORTS = ("tg_problem_create", "tg_problem_destroy", "tg_problem_info", "tg_problem_bvalues",
           "tg_enumerate_pairs", "tg_score_pairs", "tg_prune_workspace_bytes", "tg_prune",
           "tg_compose_workspace_bytes", "tg_compose_pipeline", "tg_compose_relaxed_workspace_bytes",
           "tg_compose_pipeline_relaxed", "tg_compose_all_orders_workspace_bytes",
           "tg_compose_pipeline_all_orders", "tg_build_islands_workspace_bytes", "tg_build_islands",
           "tg_score_classes", "tg_prune_classes_workspace_bytes", "tg_prune_classes",
           "tg_compose_pipeline_classes", "tg_prune_no_alloc",
           "tg_last_error")

_lib = None


def load_library(path=LIB_PATH):
    """Load the built library and declare every exported signature."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run `python -m paper_2606_16907_amd.build`")
    L = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    P = ctypes.POINTER
    L.tg_problem_create.argtypes = [P(TgLayer), i32, P(TgIsland), i32, P(ctypes.c_double),
                                    P(TgSpace), P(vp)]
    L.tg_problem_create.restype = ctypes.c_int
    L.tg_problem_destroy.argtypes = [vp]
    L.tg_problem_destroy.restype = None
    L.tg_problem_info.argtypes = [vp, P(TgInfo)]
    L.tg_problem_bvalues.argtypes = [vp, P(i64), i32]
    L.tg_enumerate_pairs.argtypes = [vp, P(i64), i64, i64, vp, vp]
    L.tg_score_pairs.argtypes = [vp, i64, i64, vp, vp, vp]
    L.tg_prune_workspace_bytes.argtypes = [vp]
    L.tg_prune_workspace_bytes.restype = sz
    L.tg_prune.argtypes = [vp, vp, vp, vp, i64, P(i64), vp, sz, vp]
    L.tg_prune_no_alloc.argtypes = [vp, vp, vp, vp, i64, P(i64), vp]
    L.tg_compose_workspace_bytes.argtypes = [vp, i64]
    L.tg_compose_workspace_bytes.restype = sz
    L.tg_compose_pipeline.argtypes = [vp, vp, i64, vp, vp, P(i32), P(TgPlan), vp, sz, vp]
    L.tg_compose_relaxed_workspace_bytes.argtypes = [vp, i64]
    L.tg_compose_relaxed_workspace_bytes.restype = sz
    L.tg_compose_pipeline_relaxed.argtypes = [vp, vp, i64, vp, vp, P(i32), P(TgPlan), vp, sz, vp]
    L.tg_compose_all_orders_workspace_bytes.argtypes = [vp, i64]
    L.tg_compose_all_orders_workspace_bytes.restype = sz
    L.tg_compose_pipeline_all_orders.argtypes = [vp, vp, i64, vp, vp, P(TgPlan), vp, sz, vp]
    L.tg_score_classes.argtypes = [vp, i64, i64, vp, vp, vp]
    L.tg_prune_classes_workspace_bytes.argtypes = [vp]
    L.tg_prune_classes_workspace_bytes.restype = sz
    L.tg_prune_classes.argtypes = [vp, vp, vp, vp, i64, P(i64), vp, sz, vp]
    L.tg_compose_pipeline_classes.argtypes = [vp, vp, i64, vp, vp, P(i32), P(TgPlan), vp, sz, vp]
    L.tg_build_islands_workspace_bytes.argtypes = [i32]
    L.tg_build_islands_workspace_bytes.restype = sz
    L.tg_build_islands.argtypes = [P(TgIsland), i32, P(ctypes.c_double), ctypes.c_double, ctypes.c_double,
                                   ctypes.c_double, P(i32), P(TgIsland), P(ctypes.c_double), P(i32), vp, sz, vp]
    L.tg_last_error.argtypes = []
    L.tg_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def last_error():
    return load_library().tg_last_error().decode()


def _check(status, what):
    if status != TG_OK:
        raise TangramError(status, what, last_error())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dbuf(t, dtype, n, what, device=None):
    """Device pointer of a caller's buffer after the checks a plain pointer
    cannot carry: a contiguous CUDA tensor of `dtype` (on `device` when one is
    given) with at least n elements.  A short buffer would be read or written
    past its end by the kernels, so it is refused here."""
    if t is None or not t.is_cuda:
        raise ValueError(f"{what}: device buffer expected")
    if t.dtype != dtype:
        raise ValueError(f"{what}: dtype {t.dtype}, {dtype} expected")
    if not t.is_contiguous():
        raise ValueError(f"{what}: contiguous buffer expected")
    if device is not None and t.device.index != device:
        raise ValueError(f"{what}: on cuda:{t.device.index}, the problem is on cuda:{device}")
    if t.numel() < n:
        raise ValueError(f"{what}: {t.numel()} elements, at least {n} needed")
    return ctypes.c_void_p(t.data_ptr())


def _dws(t, what, device=None):
    """Workspace pointer and its size in bytes (a contiguous CUDA tensor of
    any dtype; the library checks the size)."""
    if t is None or not t.is_cuda:
        raise ValueError(f"{what}: device buffer expected")
    if not t.is_contiguous():
        raise ValueError(f"{what}: contiguous buffer expected")
    if device is not None and t.device.index != device:
        raise ValueError(f"{what}: on cuda:{t.device.index}, the problem is on cuda:{device}")
    return ctypes.c_void_p(t.data_ptr()), t.numel() * t.element_size()


class Problem:
    """A planning instance resident on the current GPU (tg_problem)."""

    def __init__(self, inst):
        lib = load_library()
        lay = inst["layers"]
        L = len(lay["fwd_flops"])
        layers = (TgLayer * L)()
        for l in range(L):
            for f in LAYER_FIELDS:
                setattr(layers[l], f, int(lay[f][l]) if f in lay else 0)
        isl = inst["islands"]
        K = len(isl["n_gpus"])
        islands = (TgIsland * K)()
        for k in range(K):
            islands[k].n_gpus = int(isl["n_gpus"][k])
            islands[k].peak_flops = float(isl["peak_flops"][k])
            islands[k].hbm_bytes = float(isl["hbm_bytes"][k])
            islands[k].intra_bw = float(isl["intra_bw"][k])
            islands[k].host_bw = float(isl["host_bw"][k]) if "host_bw" in isl else 0.0
        inter = (ctypes.c_double * (K * K))(*[float(x) for row in inst["inter_bw"] for x in row])
        sp = inst["space"]
        space = TgSpace()
        space.global_batch = int(sp["global_batch"])
        space.n_experts = int(sp["n_experts"])
        for name in ("tp", "ep", "mb"):
            vals = list(sp[name])
            setattr(space, "n_" + name, len(vals))
            arr = getattr(space, name)
            for a, v in enumerate(vals[:8]):
                arr[a] = int(v)
        space.zero_mask = sum(1 << int(z) for z in sp["zero"])
        cps = list(sp.get("cp", [1]))
        space.n_cp = len(cps)
        for a, v in enumerate(cps[:8]):
            space.cp[a] = int(v)
        space.recompute_mask = sum(1 << int(r) for r in sp.get("recompute", [0]))
        space.offload_mask = sum(1 << int(r) for r in sp.get("offload", [0]))
        space.imbalance_eps = float(sp.get("imbalance_eps", 0.0))
        space.eta = float(sp["eta"])
        space.mem_frac = float(sp["mem_frac"])
        h = ctypes.c_void_p()
        _check(lib.tg_problem_create(layers, L, islands, K, inter, ctypes.byref(space),
                                     ctypes.byref(h)), "tg_problem_create")
        self.h = h
        self.inst = inst
        self.device = torch.cuda.current_device()
        info = TgInfo()
        _check(lib.tg_problem_info(self.h, ctypes.byref(info)), "tg_problem_info")
        self.L, self.K, self.n_b, self.dense = info.L, info.K, info.n_b, bool(info.dense)
        self.NS, self.n_configs, self.N = info.NS, info.n_configs, info.N
        self.n_compatible_configs = info.n_compatible_configs
        self.NC = info.n_slice_classes
        bv = (ctypes.c_int64 * max(self.n_b, 1))()
        _check(lib.tg_problem_bvalues(self.h, bv, max(self.n_b, 1)), "tg_problem_bvalues")
        self.bvalues = [int(bv[a]) for a in range(self.n_b)]

    def close(self):
        if getattr(self, "h", None) is not None and self.h.value:
            load_library().tg_problem_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # --- entry points -----------------------------------------------------
    def tg_enumerate_pairs(self, first=0, count=None, out=None):
        """Decode candidates [first, first+count) into an int32 [count, 12]
        device tensor (i, j, island, tp, cp, dp, ep, zero, recompute, offload,
        mb, 0)."""
        lib = load_library()
        n = ctypes.c_int64(0)
        if count is None:
            _check(lib.tg_enumerate_pairs(self.h, ctypes.byref(n), 0, 0, None, None),
                   "tg_enumerate_pairs")
            count = n.value - first
        if out is None:
            out = torch.empty((count, 12), dtype=torch.int32, device="cuda")
        ptr = _dbuf(out, torch.int32, 12 * int(count), "out", self.device)
        _check(lib.tg_enumerate_pairs(self.h, ctypes.byref(n), int(first), int(count), ptr,
                                      _stream()), "tg_enumerate_pairs")
        return out

    def tg_score_pairs(self, first=0, count=None, cost=None, dmax=None):
        if count is None:
            count = self.N - first
        if cost is None:
            cost = torch.empty(count, dtype=torch.float64, device="cuda")
        if dmax is None:
            dmax = torch.empty(count, dtype=torch.uint8, device="cuda")
        pc = _dbuf(cost, torch.float64, int(count), "cost", self.device)
        pd = _dbuf(dmax, torch.uint8, int(count), "dmax", self.device)
        _check(load_library().tg_score_pairs(self.h, int(first), int(count), pc, pd, _stream()),
               "tg_score_pairs")
        return cost, dmax

    # -- redundancy pruning: scores by slice class --------------------------
    def tg_score_classes(self, first=0, count=None, cost=None, dmax=None):
        if count is None:
            count = self.n_configs * self.NC - first
        if cost is None:
            cost = torch.empty(count, dtype=torch.float64, device="cuda")
        if dmax is None:
            dmax = torch.empty(count, dtype=torch.uint8, device="cuda")
        pc = _dbuf(cost, torch.float64, int(count), "cost", self.device)
        pd = _dbuf(dmax, torch.uint8, int(count), "dmax", self.device)
        _check(load_library().tg_score_classes(self.h, int(first), int(count), pc, pd, _stream()),
               "tg_score_classes")
        return cost, dmax

    def prune_classes_workspace(self):
        n = load_library().tg_prune_classes_workspace_bytes(self.h)
        return torch.empty(max(int(n), 1), dtype=torch.uint8, device="cuda")

    def tg_prune_classes(self, cost, dmax, survivors=None, workspace=None):
        """Surviving set from class scores: tg_prune's ascending list."""
        lib = load_library()
        ws = workspace if workspace is not None else self.prune_classes_workspace()
        n = ctypes.c_int64(0)
        n_scores = self.n_configs * self.NC
        pc = _dbuf(cost, torch.float64, n_scores, "cost", self.device)
        pd = _dbuf(dmax, torch.uint8, n_scores, "dmax", self.device)
        pw, wb = _dws(ws, "workspace", self.device)
        if survivors is None:
            st = lib.tg_prune_classes(self.h, pc, pd, None, 0, ctypes.byref(n), pw, wb, _stream())
            if st not in (TG_OK, TG_ECAPACITY):
                _check(st, "tg_prune_classes")
            survivors = torch.empty(max(n.value, 1), dtype=torch.int64, device="cuda")
        ps = _dbuf(survivors, torch.int64, 0, "survivors", self.device)
        st = lib.tg_prune_classes(self.h, pc, pd, ps, survivors.numel(), ctypes.byref(n), pw, wb, _stream())
        _check(st, "tg_prune_classes")
        return survivors[: n.value]

    def tg_compose_pipeline_classes(self, survivors, cost, dmax, island_order=None, workspace=None):
        """tg_compose_pipeline with class scores.  Returns (status, plan dict)."""
        lib = load_library()
        if island_order is None:
            island_order = self.inst["island_order"]
        order = (ctypes.c_int32 * self.K)(*[int(x) for x in island_order])
        n = int(survivors.numel())
        ws = workspace if workspace is not None else self.compose_workspace(n)
        plan = TgPlan()
        ps, pc, pd, pw, wb = self._compose_args(survivors, cost, dmax, ws, self.n_configs * self.NC)
        st = lib.tg_compose_pipeline_classes(self.h, ps, n, pc, pd, order, ctypes.byref(plan), pw, wb,
                                             _stream())
        if st not in (TG_OK, TG_ENOPLAN):
            _check(st, "tg_compose_pipeline_classes")
        return st, plan_to_dict(plan)

    def prune_workspace(self):
        n = load_library().tg_prune_workspace_bytes(self.h)
        return torch.empty(max(int(n), 1), dtype=torch.uint8, device="cuda")

    def tg_prune(self, cost, dmax, survivors=None, workspace=None):
        """Returns the ascending survivor list (int64 device tensor)."""
        lib = load_library()
        ws = workspace if workspace is not None else self.prune_workspace()
        n = ctypes.c_int64(0)
        pc = _dbuf(cost, torch.float64, self.N, "cost", self.device)
        pd = _dbuf(dmax, torch.uint8, self.N, "dmax", self.device)
        pw, wb = _dws(ws, "workspace", self.device)
        if survivors is None:
            st = lib.tg_prune(self.h, pc, pd, None, 0, ctypes.byref(n), pw, wb, _stream())
            if st not in (TG_OK, TG_ECAPACITY):
                _check(st, "tg_prune")
            survivors = torch.empty(max(n.value, 1), dtype=torch.int64, device="cuda")
        ps = _dbuf(survivors, torch.int64, 0, "survivors", self.device)
        st = lib.tg_prune(self.h, pc, pd, ps, survivors.numel(), ctypes.byref(n), pw, wb, _stream())
        if st == TG_ECAPACITY:
            err = TangramError(st, "tg_prune", last_error())
            err.required = n.value
            raise err
        _check(st, "tg_prune")
        return survivors[: n.value]

    def tg_prune_no_alloc(self, cost, dmax, survivors):
        """tg_prune on the library's static scratch: no workspace and no
        allocation (the caller's `survivors` buffer receives the list).
        Returns the filled prefix of `survivors`."""
        lib = load_library()
        n = ctypes.c_int64(0)
        pc = _dbuf(cost, torch.float64, self.N, "cost", self.device)
        pd = _dbuf(dmax, torch.uint8, self.N, "dmax", self.device)
        ps = _dbuf(survivors, torch.int64, 0, "survivors", self.device)
        st = lib.tg_prune_no_alloc(self.h, pc, pd, ps, survivors.numel(), ctypes.byref(n), _stream())
        if st == TG_ECAPACITY:
            err = TangramError(st, "tg_prune_no_alloc", last_error())
            err.required = n.value
            raise err
        _check(st, "tg_prune_no_alloc")
        return survivors[: n.value]

    def _compose_args(self, survivors, cost, dmax, ws, n_scores):
        """Checked pointers of a composition's survivor list, score arrays
        (n_scores entries each) and workspace."""
        n = int(survivors.numel())
        ps = _dbuf(survivors, torch.int64, n, "survivors", self.device) if n else None
        pc = _dbuf(cost, torch.float64, n_scores, "cost", self.device)
        pd = _dbuf(dmax, torch.uint8, n_scores, "dmax", self.device)
        pw, wb = _dws(ws, "workspace", self.device)
        return ps, pc, pd, pw, wb

    def compose_workspace(self, n_survivors):
        n = load_library().tg_compose_workspace_bytes(self.h, int(n_survivors))
        return torch.empty(max(int(n), 1), dtype=torch.uint8, device="cuda")

    def tg_compose_pipeline(self, survivors, cost, dmax, island_order=None, workspace=None):
        """Returns (status, plan dict)."""
        lib = load_library()
        if island_order is None:
            island_order = self.inst["island_order"]
        order = (ctypes.c_int32 * self.K)(*[int(x) for x in island_order])
        n = int(survivors.numel())
        ws = workspace if workspace is not None else self.compose_workspace(n)
        plan = TgPlan()
        ps, pc, pd, pw, wb = self._compose_args(survivors, cost, dmax, ws, self.N)
        st = lib.tg_compose_pipeline(self.h, ps, n, pc, pd, order, ctypes.byref(plan), pw, wb, _stream())
        if st not in (TG_OK, TG_ENOPLAN):
            _check(st, "tg_compose_pipeline")
        return st, plan_to_dict(plan)

    def compose_relaxed_workspace(self, n_survivors):
        n = load_library().tg_compose_relaxed_workspace_bytes(self.h, int(n_survivors))
        return torch.empty(max(int(n), 1), dtype=torch.uint8, device="cuda")

    def tg_compose_pipeline_relaxed(self, survivors, cost, dmax, island_order=None, workspace=None):
        """Composition with the step-(4) relaxation.  Returns (status, plan dict)."""
        lib = load_library()
        if island_order is None:
            island_order = self.inst["island_order"]
        order = (ctypes.c_int32 * self.K)(*[int(x) for x in island_order])
        n = int(survivors.numel())
        ws = workspace if workspace is not None else self.compose_relaxed_workspace(n)
        plan = TgPlan()
        ps, pc, pd, pw, wb = self._compose_args(survivors, cost, dmax, ws, self.N)
        st = lib.tg_compose_pipeline_relaxed(self.h, ps, n, pc, pd, order, ctypes.byref(plan), pw, wb,
                                             _stream())
        if st not in (TG_OK, TG_ENOPLAN):
            _check(st, "tg_compose_pipeline_relaxed")
        return st, plan_to_dict(plan)

    def compose_all_orders_workspace(self, n_survivors):
        n = load_library().tg_compose_all_orders_workspace_bytes(self.h, int(n_survivors))
        return torch.empty(max(int(n), 1), dtype=torch.uint8, device="cuda")

    def tg_compose_pipeline_all_orders(self, survivors, cost, dmax, workspace=None):
        """Composition over every island subset and order (K <= 16).  Returns
        (status, plan dict)."""
        lib = load_library()
        n = int(survivors.numel())
        ws = workspace if workspace is not None else self.compose_all_orders_workspace(n)
        plan = TgPlan()
        ps, pc, pd, pw, wb = self._compose_args(survivors, cost, dmax, ws, self.N)
        st = lib.tg_compose_pipeline_all_orders(self.h, ps, n, pc, pd, ctypes.byref(plan), pw, wb, _stream())
        if st not in (TG_OK, TG_ENOPLAN):
            _check(st, "tg_compose_pipeline_all_orders")
        return st, plan_to_dict(plan)

    def plan_search(self, island_order=None):
        """Score every candidate, prune, compose: the whole hot path."""
        cost, dmax = self.tg_score_pairs()
        surv = self.tg_prune(cost, dmax)
        st, plan = self.tg_compose_pipeline(surv, cost, dmax, island_order)
        return st, plan, surv, cost, dmax


def plan_to_dict(plan):
    stages = []
    for t in range(max(plan.S, 0)):
        s = plan.stage[t]
        stages.append({f: getattr(s, f) for f, _ in TgStage._fields_ if f != "reserved"})
    return {"b": plan.b, "m": plan.m, "S": plan.S, "P": plan.P, "F": plan.F, "T": plan.T,
            "stages": stages}


def build_islands(cluster, workspace=None):
    """Island construction (Sec. 4.1) of a node-level cluster (dict with
    "nodes": gpus, peak_flops, hbm_bytes, intra_bw, host_bw per node;
    "node_bw": n x n bytes/s; "eps": compute, memory, intra).  Returns
    island_of, K, islands (tg_island fields) and inter_bw (K x K)."""
    lib = load_library()
    nd = cluster["nodes"]
    n = len(nd["gpus"])
    nodes = (TgIsland * n)()
    for u in range(n):
        nodes[u].n_gpus = int(nd["gpus"][u])
        nodes[u].peak_flops = float(nd["peak_flops"][u])
        nodes[u].hbm_bytes = float(nd["hbm_bytes"][u])
        nodes[u].intra_bw = float(nd["intra_bw"][u])
        nodes[u].host_bw = float(nd["host_bw"][u])
    import numpy as np
    e_arr = np.ascontiguousarray(np.asarray(cluster["node_bw"], dtype=np.float64).reshape(n * n))
    e = e_arr.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    ws = workspace
    if ws is None:
        ws = torch.empty(max(int(lib.tg_build_islands_workspace_bytes(n)), 1), dtype=torch.uint8, device="cuda")
    isl_of = (ctypes.c_int32 * n)()
    isl = (TgIsland * n)()
    inter_arr = np.zeros(n * n, dtype=np.float64)
    inter = inter_arr.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    K = ctypes.c_int32(0)
    eps = cluster["eps"]
    st = lib.tg_build_islands(nodes, n, e, float(eps["compute"]), float(eps["memory"]), float(eps["intra"]),
                              isl_of, isl, inter, ctypes.byref(K), *_dws(ws, "workspace", torch.cuda.current_device()),
                              _stream())
    _check(st, "tg_build_islands")
    k = K.value
    return {"island_of": list(isl_of), "K": k,
            "islands": {"n_gpus": [isl[a].n_gpus for a in range(k)],
                        "peak_flops": [isl[a].peak_flops for a in range(k)],
                        "hbm_bytes": [isl[a].hbm_bytes for a in range(k)],
                        "intra_bw": [isl[a].intra_bw for a in range(k)],
                        "host_bw": [isl[a].host_bw for a in range(k)]},
            "inter_bw": inter_arr[:k * k].reshape(k, k).tolist()}
