"""Seeded synthetic planning instances: per-layer integer workloads and GPU islands.

This module only builds inputs.  It holds none of the planner's arithmetic (no
scoring, pruning or composition); both the HIP path and the CPU oracle consume
the dictionaries it returns.

Paper context (Tangram, arXiv 2606.16907):
  * model atoms are layers and a model slice is a contiguous run of atoms
    (Sec. 4.2, "Model slicing");
  * a GPU island is a homogeneous group of nodes described by GPU count,
    compute, memory and intra-node bandwidth, with inter-node bandwidth
    between islands (Sec. 4.1, Eq. 1-3).
The paper measures on GPT-3 6.7B/13B, GShard MoE and Mixtral/Qwen3 MoE models
on Azure T4/V100/A100/H100 clusters (Sec. 6.1, Tab. 3).  Those clusters and the
parallelizers' profiles cannot be reproduced here; the five instances below are
synthetic stand-ins with the shapes named in their docstrings.

Per-layer quantities are integers per sample (one sequence of length s),
forward pass, with 2-byte (bf16) activations and communication:
  fwd_flops       = 2sh(h+2h_kv) + 2sh^2 + 4s^2 h + n_mat*2shf
                    (MoE: + 2shE router + top_k*3*2sh f_e, no dense FFN)
  dense_params    = h(h+2h_kv) + h^2 + n_mat*h*f + 2h   (MoE: FFN -> h*E router)
  expert_params   = E*3*h*f_e (MoE only)
  act_stash_bytes = 10sh + 2s(h+2h_kv) + 2sh + FFN, FFN = 4sf (GeLU) / 6sf
                    (SwiGLU) / top_k*(6s f_e + 2sh) (MoE); 34sh for GPT shape
  tp_comm_bytes   = 4sh      (two s x h collectives per layer, one pass)
  a2a_bytes       = 2*(top_k*s)*h*2  (dispatch + combine, MoE only)
  out_act_bytes   = 2sh
"""
from __future__ import annotations

import json
import os

import numpy as np

LAYER_FIELDS = ("fwd_flops", "dense_params", "expert_params", "act_stash_bytes",
                "tp_comm_bytes", "a2a_bytes", "out_act_bytes", "cp_comm_bytes")
ISLAND_FIELDS = ("n_gpus", "peak_flops", "hbm_bytes", "intra_bw", "host_bw")

FIXTURE_DIR = os.path.join(os.path.dirname(os.path.abspath(__file__)), "fixtures")
CONFIG_NAMES = ("tiny", "dense8b", "dense70b", "moe", "large")


# ----------------------------------------------------------------------------
# per-layer workload
# ----------------------------------------------------------------------------
def layer_ints(s, h, n_heads, n_kv, ffn, act="gelu", n_experts=0, top_k=0, ffn_expert=0):
    """Integer per-sample quantities of one transformer layer (formulas above)."""
    d_h = h // n_heads
    h_kv = n_kv * d_h
    n_mat = 3 if act == "swiglu" else 2
    attn_flops = 2 * s * h * (h + 2 * h_kv) + 2 * s * h * h + 4 * s * s * h
    attn_params = h * (h + 2 * h_kv) + h * h + 2 * h
    attn_act = 10 * s * h + 2 * s * (h + 2 * h_kv) + 2 * s * h
    if n_experts > 0:
        fwd = attn_flops + 2 * s * h * n_experts + top_k * 3 * 2 * s * h * ffn_expert
        dense_p = attn_params + h * n_experts
        expert_p = n_experts * 3 * h * ffn_expert
        stash = attn_act + top_k * (6 * s * ffn_expert + 2 * s * h)
        a2a = 2 * (top_k * s) * h * 2
    else:
        fwd = attn_flops + n_mat * 2 * s * h * ffn
        dense_p = attn_params + n_mat * h * ffn
        expert_p = 0
        stash = attn_act + (6 if act == "swiglu" else 4) * s * ffn
        a2a = 0
    return {"fwd_flops": fwd, "dense_params": dense_p, "expert_params": expert_p,
            "act_stash_bytes": stash, "tp_comm_bytes": 4 * s * h, "a2a_bytes": a2a,
            "out_act_bytes": 2 * s * h, "cp_comm_bytes": 2 * 2 * s * h_kv}


def uniform_layers(n_layers, **shape):
    one = layer_ints(**shape)
    return {f: [int(one[f])] * n_layers for f in LAYER_FIELDS}


# ----------------------------------------------------------------------------
# islands
# ----------------------------------------------------------------------------
def host_link(hbm):
    """Host (PCIe) bandwidth per GPU, bytes/s, by GPU generation: the
    large-memory parts sit on PCIe 5 x16, the others on PCIe 4 x16.  A
    function of the drawn type, so it consumes no random numbers."""
    return 64e9 if hbm >= 100e9 else 32e9


def _draw_gpu_types(rng, n_types):
    types = []
    for _ in range(n_types):
        peak = round(float(rng.uniform(100.0, 1000.0)), 1) * 1e12
        hbm = float(rng.choice([40, 80, 141, 192])) * 1e9
        intra = round(float(rng.uniform(300.0, 900.0)), 1) * 1e9
        types.append((peak, hbm, intra))
    return types


def _canonical_order(islands, key_prefix=None):
    K = len(islands["n_gpus"])

    def key(k):
        pre = key_prefix(k) if key_prefix else ()
        return pre + (-islands["hbm_bytes"][k], -islands["peak_flops"][k],
                      -islands["n_gpus"][k], k)
    return sorted(range(K), key=key)


def random_cluster(rng, n_islands, n_types, max_nodes, one_type_per_island=False,
                   fixed_nodes=None):
    """Islands drawn per type (peak, hbm, intra), then per island (type, nodes,
    inter); E[k][k'] = min(inter_k, inter_k')."""
    types = _draw_gpu_types(rng, n_types)
    isl = {f: [] for f in ISLAND_FIELDS}
    inter = []
    for k in range(n_islands):
        t = k if one_type_per_island else int(rng.integers(0, n_types))
        nodes = fixed_nodes if fixed_nodes is not None else int(rng.integers(1, max_nodes + 1))
        peak, hbm, intra = types[t]
        isl["n_gpus"].append(8 * nodes)
        isl["peak_flops"].append(peak)
        isl["hbm_bytes"].append(hbm)
        isl["intra_bw"].append(intra)
        isl["host_bw"].append(host_link(hbm))
        inter.append(round(float(rng.uniform(12.5, 50.0)), 2) * 1e9)
    E = [[0.0 if a == b else min(inter[a], inter[b]) for b in range(n_islands)]
         for a in range(n_islands)]
    return isl, E


def fabric_cluster(rng, n_islands, n_types, max_nodes, leaf=4, spine=16,
                   bw=(400e9, 100e9, 25e9)):
    """Islands as in random_cluster, placed by a seeded permutation into leaves
    of `leaf` and spines of `spine` islands: E = bw[0] within a leaf, bw[1]
    within a spine, bw[2] otherwise."""
    types = _draw_gpu_types(rng, n_types)
    isl = {f: [] for f in ISLAND_FIELDS}
    for _ in range(n_islands):
        t = int(rng.integers(0, n_types))
        nodes = int(rng.integers(1, max_nodes + 1))
        peak, hbm, intra = types[t]
        isl["n_gpus"].append(8 * nodes)
        isl["peak_flops"].append(peak)
        isl["hbm_bytes"].append(hbm)
        isl["intra_bw"].append(intra)
        isl["host_bw"].append(host_link(hbm))
    perm = rng.permutation(n_islands)
    slot = [0] * n_islands
    for pos, k in enumerate(perm):
        slot[int(k)] = pos
    leaf_of = [slot[k] // leaf for k in range(n_islands)]
    spine_of = [slot[k] // spine for k in range(n_islands)]
    E = []
    for a in range(n_islands):
        row = []
        for b in range(n_islands):
            if a == b:
                row.append(0.0)
            elif leaf_of[a] == leaf_of[b]:
                row.append(bw[0])
            elif spine_of[a] == spine_of[b]:
                row.append(bw[1])
            else:
                row.append(bw[2])
        E.append(row)
    return isl, E, leaf_of, spine_of


def node_cluster(seed, n_nodes, n_types=5, leaf=8, pod=4, run=(4, 48), jitter=0.02,
                 bw=(400e9, 100e9, 25e9), asym=0.0, eps=(0.1, 0.1, 0.1)):
    """Node-level cluster for island construction (Sec. 4.1): nodes bought in
    batches (contiguous runs of `run` nodes of one GPU type, 8 GPUs per node),
    each node's measured compute and intra-node bandwidth within +-`jitter` of
    its type's; a leaf/pod fabric of `leaf` nodes per leaf switch and `pod`
    leaves per pod, bandwidth bw[0] inside a leaf, bw[1] inside a pod, bw[2]
    across pods, each direction of each node pair scaled by 1 + asym U[-1, 1]
    (links need not be symmetric; the default keeps each fabric level exact,
    since Eq. 3 compares link speeds without tolerance).  eps = (compute,
    memory, intra)."""
    rng = np.random.default_rng(seed)
    types = _draw_gpu_types(rng, n_types)
    t_of = []
    while len(t_of) < n_nodes:
        t = int(rng.integers(0, n_types))
        t_of += [t] * int(rng.integers(run[0], run[1] + 1))
    t_of = t_of[:n_nodes]
    nodes = {"gpus": [], "peak_flops": [], "hbm_bytes": [], "intra_bw": [], "host_bw": []}
    for u in range(n_nodes):
        peak, hbm, intra = types[t_of[u]]
        nodes["gpus"].append(8)
        nodes["peak_flops"].append(round(peak * (1.0 + jitter * float(rng.uniform(-1.0, 1.0))), -6))
        nodes["hbm_bytes"].append(hbm)
        nodes["intra_bw"].append(round(intra * (1.0 + jitter * float(rng.uniform(-1.0, 1.0))), -3))
        nodes["host_bw"].append(host_link(hbm))
    noise = rng.uniform(-1.0, 1.0, size=(n_nodes, n_nodes))
    u = np.arange(n_nodes)
    same_leaf = (u[:, None] // leaf) == (u[None, :] // leaf)
    same_pod = (u[:, None] // (leaf * pod)) == (u[None, :] // (leaf * pod))
    base = np.where(same_leaf, bw[0], np.where(same_pod, bw[1], bw[2]))
    e = np.round(base * (1.0 + asym * noise), -3)
    np.fill_diagonal(e, 0.0)
    return {"name": f"nodes{n_nodes}_s{seed}", "nodes": nodes, "node_bw": e,
            "eps": {"compute": eps[0], "memory": eps[1], "intra": eps[2]},
            "meta": {"seed": seed, "types": [list(t) for t in types], "type_of": t_of,
                     "leaf": leaf, "pod": pod}}


def _space(global_batch, tp, mb, ep=(1,), zero=(0, 1, 2, 3), n_experts=0, cp=(1,),
           recompute=(0,), offload=(0,)):
    return {"global_batch": int(global_batch), "n_experts": int(n_experts),
            "tp": list(tp), "ep": list(ep), "mb": list(mb), "zero": list(zero),
            "cp": list(cp), "recompute": list(recompute), "offload": list(offload),
            "eta": 1.0, "mem_frac": 1.0}


def extended(inst, cp=(1, 2, 4), recompute=(0, 1), offload=(0, 1)):
    """The instance with context parallelism, activation recomputation and
    offloading added to its configuration space (Sec. 2.1's parallelisms and
    memory-saving techniques as intra-island config dimensions)."""
    import copy
    out = copy.deepcopy(inst)
    out["space"]["cp"] = list(cp)
    out["space"]["recompute"] = list(recompute)
    out["space"]["offload"] = list(offload)
    out["name"] = inst.get("name", "custom") + "_ext"
    return out


# ----------------------------------------------------------------------------
# the five named instances
# ----------------------------------------------------------------------------
def make_tiny():
    """8-layer dense decoder (h 1024, 16 heads MHA, s 2048, FFN 4096 GeLU,
    global batch 64) on 2 islands of 4 GPUs: (300 TFLOP/s, 80 GB, 600 GB/s)
    and (150 TFLOP/s, 40 GB, 300 GB/s), 25 GB/s between them."""
    layers = uniform_layers(8, s=2048, h=1024, n_heads=16, n_kv=16, ffn=4096, act="gelu")
    isl = {"n_gpus": [4, 4], "peak_flops": [300e12, 150e12], "hbm_bytes": [80e9, 40e9],
           "intra_bw": [600e9, 300e9]}
    E = [[0.0, 25e9], [25e9, 0.0]]
    inst = {"name": "tiny", "layers": layers, "islands": isl, "inter_bw": E,
            "space": _space(64, tp=(1, 2, 4), mb=(1, 2, 4))}
    inst["island_order"] = _canonical_order(isl)
    inst["meta"] = {"model": "dense 8L h1024 s2048", "seed": None}
    return inst


def make_dense8b(seed=2):
    """32-layer dense (h 4096, FFN 14336 SwiGLU, 32 heads / 8 KV heads, s 4096,
    global batch 512) on 4 islands of 8 GPUs with per-island random specs."""
    rng = np.random.default_rng(seed)
    layers = uniform_layers(32, s=4096, h=4096, n_heads=32, n_kv=8, ffn=14336, act="swiglu")
    isl, E = random_cluster(rng, 4, 4, 1, one_type_per_island=True, fixed_nodes=1)
    inst = {"name": "dense8b", "layers": layers, "islands": isl, "inter_bw": E,
            "space": _space(512, tp=(1, 2, 4, 8), mb=(1, 2, 4, 8))}
    inst["island_order"] = _canonical_order(isl)
    inst["meta"] = {"model": "dense 32L h4096 SwiGLU GQA s4096", "seed": seed}
    return inst


def make_dense70b(seed=3):
    """80-layer dense (h 8192, FFN 28672 SwiGLU, 64 heads / 8 KV heads, s 8192,
    global batch 1024) on 16 islands of 8-64 GPUs drawn from 3 GPU types."""
    rng = np.random.default_rng(seed)
    layers = uniform_layers(80, s=8192, h=8192, n_heads=64, n_kv=8, ffn=28672, act="swiglu")
    isl, E = random_cluster(rng, 16, 3, 8)
    inst = {"name": "dense70b", "layers": layers, "islands": isl, "inter_bw": E,
            "space": _space(1024, tp=(1, 2, 4, 8), mb=(1, 2, 4, 8))}
    inst["island_order"] = _canonical_order(isl)
    inst["meta"] = {"model": "dense 80L h8192 SwiGLU GQA s8192", "seed": seed}
    return inst


def make_moe(seed=4):
    """48-layer MoE (h 6144, 48 heads / 8 KV heads, 64 experts top-2 with
    expert FFN 4096 SwiGLU, s 4096, global batch 2048) on 32 islands of 8-32
    GPUs across 4 GPU types; EP in {1,2,4,8,16}."""
    rng = np.random.default_rng(seed)
    layers = uniform_layers(48, s=4096, h=6144, n_heads=48, n_kv=8, ffn=0, act="swiglu",
                            n_experts=64, top_k=2, ffn_expert=4096)
    isl, E = random_cluster(rng, 32, 4, 4)
    inst = {"name": "moe", "layers": layers, "islands": isl, "inter_bw": E,
            "space": _space(2048, tp=(1, 2, 4, 8), mb=(1, 2, 4, 8), ep=(1, 2, 4, 8, 16),
                            n_experts=64)}
    inst["island_order"] = _canonical_order(isl)
    inst["meta"] = {"model": "MoE 48L h6144 64e top2 fe4096 s4096", "seed": seed}
    return inst


def make_large(seed=5):
    """128-layer dense (h 12288, FFN 49152 GeLU, 96 heads MHA, s 8192, global
    batch 4096) on 128 islands of 8-64 GPUs across 5 GPU types, inter-island
    bandwidth from a 3-level fabric (400 / 100 / 25 GB/s)."""
    rng = np.random.default_rng(seed)
    layers = uniform_layers(128, s=8192, h=12288, n_heads=96, n_kv=96, ffn=49152, act="gelu")
    isl, E, leaf_of, spine_of = fabric_cluster(rng, 128, 5, 8)
    inst = {"name": "large", "layers": layers, "islands": isl, "inter_bw": E,
            "space": _space(4096, tp=(1, 2, 4, 8), mb=(1, 2, 4, 8))}
    inst["island_order"] = _canonical_order(isl, key_prefix=lambda k: (spine_of[k], leaf_of[k]))
    inst["meta"] = {"model": "dense 128L h12288 GeLU MHA s8192", "seed": seed,
                    "leaf": leaf_of, "spine": spine_of}
    return inst


MAKERS = {"tiny": make_tiny, "dense8b": make_dense8b, "dense70b": make_dense70b,
          "moe": make_moe, "large": make_large}


def make_instance(name):
    return MAKERS[name]()


def random_tiny(seed, L_range=(2, 6), K_range=(1, 3), tight=False):
    """Small random instance with non-uniform layers, for exhaustive checks.

    Layers are random integers; islands have 1-4 GPUs; some inter-island links
    are zero (no link).  `tight` scales memory down so depth limits bind."""
    rng = np.random.default_rng(seed)
    L = int(rng.integers(L_range[0], L_range[1] + 1))
    K = int(rng.integers(K_range[0], K_range[1] + 1))
    moe = bool(rng.integers(0, 4) == 0)
    layers = {f: [] for f in LAYER_FIELDS}
    for _ in range(L):
        layers["fwd_flops"].append(int(rng.integers(1, 1000)) * 10**9)
        layers["dense_params"].append(int(rng.integers(1, 250)) * 10**6)
        layers["expert_params"].append(int(rng.integers(0, 250)) * 10**6 if moe else 0)
        layers["act_stash_bytes"].append(int(rng.integers(0, 400)) * 10**6)
        layers["tp_comm_bytes"].append(int(rng.integers(0, 100)) * 10**6)
        layers["a2a_bytes"].append(int(rng.integers(0, 100)) * 10**6 if moe else 0)
        layers["out_act_bytes"].append(int(rng.integers(0, 100)) * 10**6)
        layers["cp_comm_bytes"].append(layers["tp_comm_bytes"][-1])  # no extra draw
    isl = {f: [] for f in ISLAND_FIELDS}
    for _ in range(K):
        isl["n_gpus"].append(int(rng.integers(1, 5)))
        isl["peak_flops"].append(float(rng.integers(50, 500)) * 1e12)
        mem = float(rng.integers(4, 64)) * 1e9
        if tight:
            mem = mem / 4.0
        isl["hbm_bytes"].append(mem)
        isl["intra_bw"].append(float(rng.integers(50, 500)) * 1e9)
        isl["host_bw"].append(16e9)  # no extra draw
    E = [[0.0] * K for _ in range(K)]
    for a in range(K):
        for b in range(K):
            if a != b:
                E[a][b] = 0.0 if rng.integers(0, 5) == 0 else float(rng.integers(5, 100)) * 1e9
    B = int(rng.choice([4, 6, 8, 12]))
    space = _space(B, tp=(1, 2), mb=(1, 2), ep=(1, 2) if moe else (1,),
                   zero=tuple(sorted(set(int(z) for z in rng.choice(4, size=2, replace=True)) | {0})),
                   n_experts=4 if moe else 0)
    order = [int(x) for x in rng.permutation(K)]
    return {"name": f"rand{seed}", "layers": layers, "islands": isl, "inter_bw": E,
            "space": space, "island_order": order, "meta": {"seed": seed, "tight": tight}}


# ----------------------------------------------------------------------------
# fixtures
# ----------------------------------------------------------------------------
def fixture_path(name):
    return os.path.join(FIXTURE_DIR, f"{name}.json")


def dumps(inst):
    return json.dumps(inst, sort_keys=True, separators=(",", ":"))


def load_instance(name):
    with open(fixture_path(name)) as fh:
        return json.load(fh)


def write_fixtures():
    os.makedirs(FIXTURE_DIR, exist_ok=True)
    for name in CONFIG_NAMES:
        with open(fixture_path(name), "w") as fh:
            fh.write(dumps(make_instance(name)))
            fh.write("\n")


if __name__ == "__main__":
    write_fixtures()
    for name in CONFIG_NAMES:
        inst = load_instance(name)
        print(name, "L", len(inst["layers"]["fwd_flops"]), "K", len(inst["islands"]["n_gpus"]))
