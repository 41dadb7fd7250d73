"""Seeded instances at the edges of the supported sizes: up to 255 islands
(every padded island-count class of the composition kernels), up to 512
layers, link tables with few distinct bandwidths and with more than 256 of
them, and a one-island case.  Layers and islands are random (non-uniform);
the config grid is kept small so the oracle finishes in seconds."""
from __future__ import annotations

import numpy as np

from workloads import LAYER_FIELDS


def wide_instance(seed, K, L, distinct_links, B=None, tight=False):
    """Long models (L > 64) get small layers, a global batch of 1024 (many
    micro-batches, so the relaxed search has narrow windows) and no memory cut."""
    rng = np.random.default_rng(seed)
    if B is None:
        B = 8 if L <= 64 else 1024
    tight = tight and L <= 64
    layers = {f: [] for f in LAYER_FIELDS}
    unit = 10**6 if L <= 64 else 10**4  # long models get small layers so plans fit
    for _ in range(L):
        layers["fwd_flops"].append(int(rng.integers(1, 1000)) * 10**9)
        layers["dense_params"].append(int(rng.integers(1, 250)) * unit)
        layers["expert_params"].append(0)
        layers["act_stash_bytes"].append(int(rng.integers(0, 400)) * unit)
        layers["tp_comm_bytes"].append(int(rng.integers(0, 100)) * 10**6)
        layers["a2a_bytes"].append(0)
        layers["out_act_bytes"].append(int(rng.integers(1, 100)) * 10**6)
        layers["cp_comm_bytes"].append(layers["tp_comm_bytes"][-1])  # no extra draw
    # a few GPU types, so islands repeat specs as in real clusters
    types = [(float(rng.integers(50, 500)) * 1e12, float(rng.integers(4, 64)) * 1e9,
              float(rng.integers(50, 500)) * 1e9) for _ in range(5)]
    isl = {"n_gpus": [], "peak_flops": [], "hbm_bytes": [], "intra_bw": [], "host_bw": []}
    for _ in range(K):
        t = types[int(rng.integers(0, len(types)))]
        isl["n_gpus"].append(int(rng.integers(1, 5)))
        isl["peak_flops"].append(t[0])
        isl["hbm_bytes"].append(t[1] / (4.0 if tight else 1.0))
        isl["intra_bw"].append(t[2])
        isl["host_bw"].append(32e9)
    if distinct_links == "few":
        levels = [400e9, 100e9, 25e9]
        E = [[0.0 if a == b else levels[int(rng.integers(0, 3))] for b in range(K)] for a in range(K)]
    else:
        E = [[0.0 if a == b else float(rng.integers(5, 5000)) * 1e7 for b in range(K)] for a in range(K)]
    # some missing links
    for a in range(K):
        for b in range(K):
            if a != b and rng.integers(0, 7) == 0:
                E[a][b] = 0.0
    space = {"global_batch": B, "n_experts": 0, "tp": [1, 2], "ep": [1], "mb": [1, 2],
             "zero": [0, 3], "eta": 1.0, "mem_frac": 1.0}
    order = [int(x) for x in rng.permutation(K)]
    return {"name": f"wide{seed}_K{K}_L{L}", "layers": layers, "islands": isl, "inter_bw": E,
            "space": space, "island_order": order, "meta": {"seed": seed}}


# (seed, K, L, links): K crosses every padded class boundary (64, 128, 192,
# 256) and the distinct-bandwidth table limit; L reaches the maximum of 512
EDGE_CASES = [
    (1, 64, 9, "few"), (2, 65, 6, "many"), (3, 128, 8, "few"), (4, 129, 4, "many"),
    (5, 192, 7, "few"), (6, 193, 4, "many"), (7, 255, 12, "few"), (8, 255, 4, "many"),
    (9, 2, 512, "few"), (10, 1, 512, "few"), (11, 3, 300, "many"),
]
