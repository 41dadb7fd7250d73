"""ctypes wrapper of the plain C oracle (tangram_oracle.c).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg.  The product path never imports this module.

Each function states which part of the plan search it checks; the C file holds
the definitions and their paper citations (Sec. 4.2 slices, Sec. 5.1 pruning,
Sec. 5.2 composition).  Inputs are the instance dictionaries of `workloads`.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "tangram_oracle.c")
# TG_ORACLE_LIB names a separately built copy (the sanitizer run builds one
# with AddressSanitizer and UndefinedBehaviorSanitizer); build() leaves it as is
LIB_OVERRIDE = os.environ.get("TG_ORACLE_LIB")
LIB = LIB_OVERRIDE or os.path.join(HERE, "libtg_oracle.so")
CFLAGS = ["-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", "-Wall",
          "-Wno-unused-function"]

LAYER_FIELDS = ("fwd_flops", "dense_params", "expert_params", "act_stash_bytes",
                "tp_comm_bytes", "a2a_bytes", "out_act_bytes", "cp_comm_bytes")
# instance keys added with context parallelism, recomputation and offloading;
# instances without them use these values
LAYER_DEFAULT = 0           # per-layer field absent: zeros
HOST_BW_DEFAULT = 0.0       # no host link: offloading not admitted
SPACE_DEFAULTS = {"cp": [1], "recompute": [0], "offload": [0], "imbalance_eps": 0.0}

OK, EINVAL, ENOMEM, ECAPACITY, ENOPLAN = 0, -1, -2, -4, -5


def build(force=True, out=None, extra=()):
    """Compile the oracle with gcc: -O2, no FMA contraction, no fast-math.
    `out` and `extra` build another copy (e.g. with sanitizers) elsewhere."""
    if out is None:
        if LIB_OVERRIDE:
            return LIB
        out = LIB
        if not force and os.path.exists(out) and os.path.getmtime(out) >= os.path.getmtime(SRC):
            return out
    tmp = out + ".tmp"
    subprocess.check_call(["gcc"] + CFLAGS + list(extra) + ["-o", tmp, SRC, "-lm"])
    os.replace(tmp, out)
    return out


class Stage(ctypes.Structure):
    _fields_ = [("island", ctypes.c_int32), ("first_layer", ctypes.c_int32),
                ("end_layer", ctypes.c_int32), ("tp", ctypes.c_int32), ("cp", ctypes.c_int32),
                ("dp", ctypes.c_int32), ("ep", ctypes.c_int32), ("zero", ctypes.c_int32),
                ("recompute", ctypes.c_int32), ("offload", ctypes.c_int32), ("mb", ctypes.c_int32),
                ("depth", ctypes.c_int32),
                ("pair_index", ctypes.c_int64), ("cost", ctypes.c_double),
                ("mem_bytes", ctypes.c_double), ("link_out", ctypes.c_double)]


class Plan(ctypes.Structure):
    _fields_ = [("status", ctypes.c_int32), ("b", ctypes.c_int32), ("m", ctypes.c_int32),
                ("S", ctypes.c_int32), ("P", ctypes.c_double), ("F", ctypes.c_double),
                ("T", ctypes.c_double), ("stage", Stage * 255)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(LIB)
        vp = ctypes.c_void_p
        i64p = ctypes.POINTER(ctypes.c_int64)
        i32p = ctypes.POINTER(ctypes.c_int32)
        f64p = ctypes.POINTER(ctypes.c_double)
        u8p = ctypes.POINTER(ctypes.c_uint8)
        L.tgo_create.argtypes = [i64p, ctypes.c_int, i32p, f64p, f64p, f64p, f64p, ctypes.c_int, f64p,
                                 ctypes.c_int64, ctypes.c_int, i32p, ctypes.c_int, i32p, ctypes.c_int,
                                 i32p, ctypes.c_int, i32p, ctypes.c_int, ctypes.c_uint32,
                                 ctypes.c_uint32, ctypes.c_uint32, ctypes.c_double, ctypes.c_double,
                                 ctypes.c_double, ctypes.POINTER(vp)]
        L.tgo_destroy.argtypes = [vp]
        L.tgo_counts.argtypes = [vp, i64p]
        L.tgo_bvalues.argtypes = [vp, i64p]
        L.tgo_decode.argtypes = [vp, ctypes.c_int64, i32p]
        L.tgo_coef.argtypes = [vp, ctypes.c_int64, f64p]
        L.tgo_score.argtypes = [vp, ctypes.c_int64, ctypes.c_int64, f64p, u8p]
        L.tgo_score_list.argtypes = [vp, i64p, ctypes.c_int64, f64p, u8p]
        L.tgo_prune.argtypes = [vp, i64p, ctypes.c_int64, i64p]
        L.tgo_compose.argtypes = [vp, i64p, ctypes.c_int64, i32p, ctypes.POINTER(Plan), f64p]
        L.tgo_compose_relaxed.argtypes = [vp, i64p, ctypes.c_int64, i32p, ctypes.POINTER(Plan), f64p]
        L.tgo_compose_all_orders.argtypes = [vp, i64p, ctypes.c_int64, ctypes.POINTER(Plan), f64p]
        L.tgo_balanced.argtypes = [vp, ctypes.c_int64, ctypes.c_int]
        _lib = L
    return _lib


def _ptr(a, ct):
    return a.ctypes.data_as(ctypes.POINTER(ct))


class OracleError(RuntimeError):
    def __init__(self, status, what):
        super().__init__(f"oracle {what} failed with status {status}")
        self.status = status


class Oracle:
    """One planning instance held by the oracle."""

    def __init__(self, inst):
        self.inst = inst
        L0 = len(inst["layers"]["fwd_flops"])
        lay = np.array([inst["layers"].get(f, [LAYER_DEFAULT] * L0) for f in LAYER_FIELDS],
                       dtype=np.int64)
        self.L = lay.shape[1]
        isl = inst["islands"]
        self.K = len(isl["n_gpus"])
        sp = inst["space"]
        n_gpus = np.array(isl["n_gpus"], dtype=np.int32)
        peak = np.array(isl["peak_flops"], dtype=np.float64)
        hbm = np.array(isl["hbm_bytes"], dtype=np.float64)
        intra = np.array(isl["intra_bw"], dtype=np.float64)
        host = np.array(isl.get("host_bw", [HOST_BW_DEFAULT] * self.K), dtype=np.float64)
        inter = np.ascontiguousarray(np.array(inst["inter_bw"], dtype=np.float64).reshape(-1))
        tp = np.array(sp["tp"], dtype=np.int32)
        ep = np.array(sp["ep"], dtype=np.int32)
        mb = np.array(sp["mb"], dtype=np.int32)
        cp = np.array(sp.get("cp", SPACE_DEFAULTS["cp"]), dtype=np.int32)
        zmask = rmask = omask = 0
        for z in sp["zero"]:
            zmask |= 1 << int(z)
        for r in sp.get("recompute", SPACE_DEFAULTS["recompute"]):
            rmask |= 1 << int(r)
        for r in sp.get("offload", SPACE_DEFAULTS["offload"]):
            omask |= 1 << int(r)
        self._keep = (lay, n_gpus, peak, hbm, intra, host, inter, tp, cp, ep, mb)
        h = ctypes.c_void_p()
        st = lib().tgo_create(_ptr(lay, ctypes.c_int64), self.L, _ptr(n_gpus, ctypes.c_int32),
                              _ptr(peak, ctypes.c_double), _ptr(hbm, ctypes.c_double),
                              _ptr(intra, ctypes.c_double), _ptr(host, ctypes.c_double), self.K,
                              _ptr(inter, ctypes.c_double), int(sp["global_batch"]),
                              int(sp["n_experts"]), _ptr(tp, ctypes.c_int32), len(tp),
                              _ptr(cp, ctypes.c_int32), len(cp), _ptr(ep, ctypes.c_int32), len(ep),
                              _ptr(mb, ctypes.c_int32), len(mb), zmask, rmask, omask,
                              float(sp["eta"]), float(sp["mem_frac"]),
                              float(sp.get("imbalance_eps", SPACE_DEFAULTS["imbalance_eps"])), ctypes.byref(h))
        if st != OK:
            raise OracleError(st, "create")
        self.h = h
        c = np.zeros(4, dtype=np.int64)
        lib().tgo_counts(self.h, _ptr(c, ctypes.c_int64))
        self.NS, self.n_configs, self.N, self.n_b = (int(x) for x in c)
        bv = np.zeros(max(self.n_b, 1), dtype=np.int64)
        lib().tgo_bvalues(self.h, _ptr(bv, ctypes.c_int64))
        self.bvalues = [int(x) for x in bv[: self.n_b]]

    def __del__(self):
        h = getattr(self, "h", None)
        if h is not None and h.value:
            lib().tgo_destroy(h)
            self.h = None

    # -- candidate space ---------------------------------------------------
    def decode(self, idx):
        out = np.zeros(11, dtype=np.int32)
        st = lib().tgo_decode(self.h, int(idx), _ptr(out, ctypes.c_int32))
        if st != OK:
            raise OracleError(st, "decode")
        i, j, k, tp, cp, dp, ep, z, rc, of, mb = (int(x) for x in out)
        return dict(i=i, j=j, island=k, tp=tp, cp=cp, dp=dp, ep=ep, zero=z, recompute=rc,
                    offload=of, mb=mb)

    def coef(self, g):
        out = np.zeros(12, dtype=np.float64)
        st = lib().tgo_coef(self.h, int(g), _ptr(out, ctypes.c_double))
        if st != OK:
            raise OracleError(st, "coef")
        names = ("alpha", "beta", "gamma", "delta_d", "delta_e", "mu_d", "mu_e", "rho", "H", "m_real",
                 "kappa", "omega")
        return dict(zip(names, (float(x) for x in out)))

    # -- scoring -----------------------------------------------------------
    def score(self, first=0, count=None):
        if count is None:
            count = self.N - first
        cost = np.empty(count, dtype=np.float64)
        dmax = np.empty(count, dtype=np.uint8)
        st = lib().tgo_score(self.h, int(first), int(count), _ptr(cost, ctypes.c_double),
                             _ptr(dmax, ctypes.c_uint8))
        if st != OK:
            raise OracleError(st, "score")
        return cost, dmax

    def score_list(self, idx):
        idx = np.ascontiguousarray(np.asarray(idx, dtype=np.int64))
        cost = np.empty(len(idx), dtype=np.float64)
        dmax = np.empty(len(idx), dtype=np.uint8)
        st = lib().tgo_score_list(self.h, _ptr(idx, ctypes.c_int64), len(idx),
                                  _ptr(cost, ctypes.c_double), _ptr(dmax, ctypes.c_uint8))
        if st != OK:
            raise OracleError(st, "score_list")
        return cost, dmax

    # -- pruning -----------------------------------------------------------
    def balanced(self, i, j, island):
        """Whether slice [i, j) on `island` passes imbalance pruning."""
        s = i * self.L - (i * (i - 1)) // 2 + (j - i - 1)
        r = lib().tgo_balanced(self.h, s, int(island))
        if r < 0:
            raise OracleError(r, "balanced")
        return bool(r)

    def slice_classes(self):
        """Class of every slice (equal per-slice sums), numbered by first slice."""
        cls = np.zeros(self.NS, dtype=np.int32)
        n = ctypes.c_int64(0)
        L_ = lib()
        L_.tgo_slice_classes.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32),
                                         ctypes.POINTER(ctypes.c_int64)]
        st = L_.tgo_slice_classes(self.h, _ptr(cls, ctypes.c_int32), ctypes.byref(n))
        if st != OK:
            raise OracleError(st, "slice_classes")
        return cls, n.value

    def prune_classes(self):
        """The surviving set computed with redundancy pruning (one staircase
        per slice class, copied to the class's slices)."""
        L_ = lib()
        L_.tgo_prune_classes.argtypes = [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int64), ctypes.c_int64,
                                         ctypes.POINTER(ctypes.c_int64)]
        n = ctypes.c_int64(0)
        st = L_.tgo_prune_classes(self.h, None, 0, ctypes.byref(n))
        if st not in (OK, ECAPACITY):
            raise OracleError(st, "prune_classes")
        out = np.zeros(max(n.value, 1), dtype=np.int64)
        st = L_.tgo_prune_classes(self.h, _ptr(out, ctypes.c_int64), n.value, ctypes.byref(n))
        if st != OK:
            raise OracleError(st, "prune_classes")
        return out[: n.value]

    def prune(self):
        n = ctypes.c_int64(0)
        lib().tgo_prune(self.h, None, 0, ctypes.byref(n))
        out = np.empty(max(n.value, 1), dtype=np.int64)
        st = lib().tgo_prune(self.h, _ptr(out, ctypes.c_int64), len(out), ctypes.byref(n))
        if st != OK:
            raise OracleError(st, "prune")
        return out[: n.value]

    # -- composition -------------------------------------------------------
    def compose(self, candidates, order=None):
        """Returns (status, plan dict, per-b array [n_b, 3] of P*, F*, T)."""
        if order is None:
            order = self.inst["island_order"]
        cands = np.ascontiguousarray(np.asarray(candidates, dtype=np.int64))
        order = np.ascontiguousarray(np.asarray(order, dtype=np.int32))
        plan = Plan()
        per_b = np.full((max(self.n_b, 1), 3), np.inf)
        st = lib().tgo_compose(self.h, _ptr(cands, ctypes.c_int64), len(cands),
                               _ptr(order, ctypes.c_int32), ctypes.byref(plan),
                               _ptr(per_b, ctypes.c_double))
        return st, plan_to_dict(plan), per_b[: self.n_b]

    def compose_relaxed(self, candidates, order=None):
        """Composition with the relaxation of step (4).  Returns (status, plan
        dict, per-b array [n_b, 4] of P*, chosen bound, F at it, T)."""
        if order is None:
            order = self.inst["island_order"]
        cands = np.ascontiguousarray(np.asarray(candidates, dtype=np.int64))
        order = np.ascontiguousarray(np.asarray(order, dtype=np.int32))
        plan = Plan()
        per_b = np.full((max(self.n_b, 1), 4), np.inf)
        st = lib().tgo_compose_relaxed(self.h, _ptr(cands, ctypes.c_int64), len(cands),
                                       _ptr(order, ctypes.c_int32), ctypes.byref(plan),
                                       _ptr(per_b, ctypes.c_double))
        return st, plan_to_dict(plan), per_b[: self.n_b]

    def compose_all_orders(self, candidates):
        """Composition over every island subset and order (steps (1)-(3); no
        order input; K <= 16).  Returns (status, plan dict, per-b array [n_b, 3]
        of P*, F*, T)."""
        cands = np.ascontiguousarray(np.asarray(candidates, dtype=np.int64))
        plan = Plan()
        per_b = np.full((max(self.n_b, 1), 3), np.inf)
        st = lib().tgo_compose_all_orders(self.h, _ptr(cands, ctypes.c_int64), len(cands), ctypes.byref(plan),
                                    _ptr(per_b, ctypes.c_double))
        return st, plan_to_dict(plan), per_b[: self.n_b]


def plan_to_dict(plan):
    stages = []
    for t in range(max(plan.S, 0)):
        s = plan.stage[t]
        stages.append({f: getattr(s, f) for f, _ in Stage._fields_})
    return {"status": plan.status, "b": plan.b, "m": plan.m, "S": plan.S, "P": plan.P,
            "F": plan.F, "T": plan.T, "stages": stages}


def build_islands(cluster):
    """Island construction (Sec. 4.1) of a node-level cluster: dict with
    "nodes" (gpus, peak_flops, hbm_bytes, intra_bw, host_bw per node),
    "node_bw" (n x n bytes/s, row = source) and "eps" (compute, memory,
    intra).  Returns island_of (per node), K, islands (the tg_island fields)
    and inter_bw (K x K)."""
    nd = cluster["nodes"]
    n = len(nd["gpus"])
    gpus = np.ascontiguousarray(np.array(nd["gpus"], dtype=np.int32))
    cols = [np.ascontiguousarray(np.array(nd[f], dtype=np.float64))
            for f in ("peak_flops", "hbm_bytes", "intra_bw", "host_bw")]
    e = np.ascontiguousarray(np.array(cluster["node_bw"], dtype=np.float64).reshape(-1))
    eps = cluster["eps"]
    isl = np.zeros(n, dtype=np.int32)
    K = ctypes.c_int32(0)
    og = np.zeros(n, dtype=np.int32)
    out = [np.zeros(n, dtype=np.float64) for _ in range(4)]
    oe = np.zeros(n * n, dtype=np.float64)
    L_ = lib()
    f = L_.tgo_build_islands
    f.argtypes = [ctypes.POINTER(ctypes.c_int32)] + [ctypes.POINTER(ctypes.c_double)] * 4 + [
        ctypes.c_int, ctypes.POINTER(ctypes.c_double), ctypes.c_double, ctypes.c_double, ctypes.c_double,
        ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32)] + [
        ctypes.POINTER(ctypes.c_double)] * 5
    st = f(_ptr(gpus, ctypes.c_int32), *[_ptr(x, ctypes.c_double) for x in cols], n,
           _ptr(e, ctypes.c_double), float(eps["compute"]), float(eps["memory"]), float(eps["intra"]),
           _ptr(isl, ctypes.c_int32), ctypes.byref(K), _ptr(og, ctypes.c_int32),
           *[_ptr(x, ctypes.c_double) for x in out], _ptr(oe, ctypes.c_double))
    if st != OK:
        raise OracleError(st, "build_islands")
    k = K.value
    return {"island_of": isl.tolist(), "K": k,
            "islands": {"n_gpus": og[:k].tolist(), "peak_flops": out[0][:k].tolist(),
                        "hbm_bytes": out[1][:k].tolist(), "intra_bw": out[2][:k].tolist(),
                        "host_bw": out[3][:k].tolist()},
            "inter_bw": oe[:k * k].reshape(k, k).tolist()}
