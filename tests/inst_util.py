"""Hand-built planning instances for closed-form and behavioural checks."""
from __future__ import annotations

import copy

from workloads import LAYER_FIELDS


def instance(L=1, K=1, layer=None, layers=None, n_gpus=1, peak=2.0**40, hbm=2.0**50,
             intra=2.0**30, inter=25e9, B=1, tp=(1,), ep=(1,), mb=(1,), zero=(0,),
             n_experts=0, order=None, eta=1.0, mem_frac=1.0, host=0.0, cp=(1,), recompute=(0,),
             offload=(0,)):
    """Instance with L identical layers (or explicit `layers`) and K islands.

    Scalars for island fields apply to every island; lists give per-island
    values.  `inter` is a scalar (all pairs) or a K x K matrix."""
    if layers is None:
        base = {f: 0 for f in LAYER_FIELDS}
        base.update(layer or {})
        layers = {f: [int(base[f])] * L for f in LAYER_FIELDS}
    else:
        L = len(layers["fwd_flops"])
        layers = {f: [int(v) for v in layers.get(f, [0] * L)] for f in LAYER_FIELDS}

    def per(v, cast):
        return [cast(x) for x in v] if isinstance(v, (list, tuple)) else [cast(v)] * K

    isl = {"n_gpus": per(n_gpus, int), "peak_flops": per(peak, float),
           "hbm_bytes": per(hbm, float), "intra_bw": per(intra, float), "host_bw": per(host, float)}
    if isinstance(inter, (list, tuple)):
        E = [[float(x) for x in row] for row in inter]
    else:
        E = [[0.0 if a == b else float(inter) for b in range(K)] for a in range(K)]
    return {"name": "custom", "layers": layers, "islands": isl, "inter_bw": E,
            "space": {"global_batch": int(B), "n_experts": int(n_experts), "tp": list(tp),
                      "ep": list(ep), "mb": list(mb), "zero": list(zero), "cp": list(cp),
                      "recompute": list(recompute), "offload": list(offload), "eta": float(eta),
                      "mem_frac": float(mem_frac)},
            "island_order": list(order) if order is not None else list(range(K)),
            "meta": {}}


def scaled(inst, compute=1.0, bandwidth=1.0, memory=1.0):
    out = copy.deepcopy(inst)
    isl = out["islands"]
    isl["peak_flops"] = [x * compute for x in isl["peak_flops"]]
    isl["intra_bw"] = [x * bandwidth for x in isl["intra_bw"]]
    isl["hbm_bytes"] = [x * memory for x in isl["hbm_bytes"]]
    if "host_bw" in isl:
        isl["host_bw"] = [x * bandwidth for x in isl["host_bw"]]
    out["inter_bw"] = [[x * bandwidth for x in row] for row in out["inter_bw"]]
    return out


def tiny_tight():
    """The tiny dense instance with HBM cut so pipeline depth limits bind."""
    from workloads import make_instance
    inst = make_instance("tiny")
    inst = scaled(inst, memory=1.0 / 16.0)
    inst["name"] = "tiny_tight"
    return inst
