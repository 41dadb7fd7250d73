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


def deep_staircase(seed):
    """Mixture-of-experts instance on 8 islands of 8 GPUs with at most 32
    configs per (island, micro-batch) group, where the expert-parallel degrees
    give some (slice, island, b) groups five or six survivors (seeds 105, 111,
    123 and 135 do)."""
    import numpy as np
    rng = np.random.default_rng(seed)
    L, K = int(rng.integers(3, 7)), 8
    layers = {"fwd_flops": [int(rng.integers(100, 1000)) * 10**9 for _ in range(L)],
              "dense_params": [int(rng.integers(10, 100)) * 10**6 for _ in range(L)],
              "expert_params": [int(rng.integers(200, 2000)) * 10**6 for _ in range(L)],
              "act_stash_bytes": [int(rng.integers(100, 2000)) * 10**6 for _ in range(L)],
              "tp_comm_bytes": [int(rng.integers(10, 200)) * 10**6 for _ in range(L)],
              "a2a_bytes": [int(rng.integers(10, 400)) * 10**6 for _ in range(L)],
              "out_act_bytes": [int(rng.integers(10, 100)) * 10**6 for _ in range(L)]}
    hbm = [float(rng.integers(4, 60)) * 1e9 for _ in range(K)]
    inst = instance(K=K, layers=layers, n_gpus=8, peak=[float(rng.integers(100, 900)) * 1e12 for _ in range(K)],
                    hbm=hbm, intra=[float(rng.integers(100, 900)) * 1e9 for _ in range(K)], inter=50e9, B=64,
                    tp=(1, 2), ep=(1, 2, 4, 8), mb=(1, 2, 4, 8), zero=(0, 3), n_experts=8)
    inst["name"] = f"deep_staircase{seed}"
    return inst


def longest_staircase(oracle, survivors):
    """Most survivors in one (slice, island, b) group, and the most
    compatible configs in one (island, b) group."""
    import collections
    NS, B = oracle.NS, oracle.inst["space"]["global_batch"]
    key = {}
    for g in range(oracle.n_configs):
        d = oracle.decode(g * NS)
        key[g] = (d["island"], d["dp"] * d["mb"])
    groups = collections.Counter((int(x) % NS, key[int(x) // NS]) for x in survivors)
    members = collections.Counter(k for k in key.values() if B % k[1] == 0)
    return max(groups.values(), default=0), max(members.values(), default=0)
