"""Pins of the oracle's island construction (Sec. 4.1): every island it
returns meets the island definition (same GPUs per node, Eq. 1 compute and
memory ratios, Eq. 2 intra-node bandwidth ratio, Eq. 3 links inside at least
as fast as links leaving, each checked pair by pair); no two islands of one
step-(2) group can be merged (step (3) stops only when every merge breaks
Eq. 3); closed forms on hand-built fabrics; the island attributes and
island-to-island bandwidth as sums and minima over members."""
import itertools
import math

import numpy as np
import pytest

from oracle.oracle import OracleError, EINVAL, build_islands
from workloads import node_cluster


def cluster(gpus, peak, e, hbm=None, intra=None, host=None, eps=(0.1, 0.1, 0.1)):
    n = len(gpus)
    return {"nodes": {"gpus": list(gpus), "peak_flops": list(peak),
                      "hbm_bytes": list(hbm or [80e9] * n), "intra_bw": list(intra or [600e9] * n),
                      "host_bw": list(host or [64e9] * n)},
            "node_bw": e, "eps": {"compute": eps[0], "memory": eps[1], "intra": eps[2]}}


def fabric(n, leaf, pod, bw=(400e9, 100e9, 25e9)):
    return [[0.0 if u == v else (bw[0] if u // leaf == v // leaf else
                                 (bw[1] if u // (leaf * pod) == v // (leaf * pod) else bw[2]))
             for v in range(n)] for u in range(n)]


def members(r):
    out = {}
    for u, k in enumerate(r["island_of"]):
        out.setdefault(k, []).append(u)
    return [out[k] for k in range(r["K"])]


def eq3(e, I, n):
    for u in I:
        inside = [e[u][v] for v in I if v != u]
        outside = [e[u][w] for w in range(n) if w not in I]
        if inside and outside and min(inside) < max(outside):
            return False
    return True


def within(vals, eps):
    return all(max(a, b) / min(a, b) <= 1 + eps + 1e-12 for a, b in itertools.combinations(vals, 2))


def groups_of_steps_1_2(cl):
    """Node groups after steps (1)-(2), by the stated sweep (for the
    maximality check only)."""
    nd, eps = cl["nodes"], cl["eps"]
    n = len(nd["gpus"])
    grp = [0] * n
    for field, tol in (("gpus", 0.0), ("peak_flops", eps["compute"]), ("hbm_bytes", eps["memory"]),
                       ("intra_bw", eps["intra"])):
        order = sorted(range(n), key=lambda u: (grp[u], float(nd[field][u]), u))
        new, g, v0, prev = [0] * n, -1, 0.0, None
        for u in order:
            v = float(nd[field][u])
            if prev is None or grp[u] != prev or not (v <= v0 * (1.0 + tol)):
                g, v0 = g + 1, v
            prev = grp[u]
            new[u] = g
        grp = new
    return grp


CLUSTERS = [(f"seed{s}_n{n}", s, n) for s, n in itertools.product(range(6), (12, 24, 40))]


@pytest.mark.parametrize("name,seed,n", CLUSTERS, ids=[c[0] for c in CLUSTERS])
def test_islands_meet_the_definition_and_are_maximal(name, seed, n):
    cl = node_cluster(seed, n, n_types=3, leaf=4, pod=2, run=(2, 9), asym=0.0 if seed % 2 else 0.01)
    r = build_islands(cl)
    nd, eps, e = cl["nodes"], cl["eps"], cl["node_bw"]
    isl = members(r)
    assert sorted(u for I in isl for u in I) == list(range(n))
    for I in isl:
        assert len({nd["gpus"][u] for u in I}) == 1
        assert within([nd["peak_flops"][u] for u in I], eps["compute"])
        assert within([nd["hbm_bytes"][u] for u in I], eps["memory"])
        assert within([nd["intra_bw"][u] for u in I], eps["intra"])
        assert eq3(e, I, n)
    grp = groups_of_steps_1_2(cl)
    for A, B in itertools.combinations(isl, 2):
        if grp[A[0]] == grp[B[0]]:
            assert not eq3(e, A + B, n), (A, B)
    # islands numbered by their smallest node
    assert [min(I) for I in isl] == sorted(min(I) for I in isl)


def test_homogeneous_cluster_is_one_island_whatever_the_fabric():
    n = 16
    r = build_islands(cluster([8] * n, [300e12] * n, fabric(n, 4, 2)))
    assert r["K"] == 1 and r["islands"]["n_gpus"] == [8 * n]


def test_compute_tolerance_splits_by_sweep():
    # 100, 105 | 112, 120 with eps_c = 0.1: 112 > 100 * 1.1 opens a group, 120 <= 112 * 1.1
    peak = [100e12, 112e12, 105e12, 120e12]
    r = build_islands(cluster([8] * 4, peak, fabric(4, 4, 1)))
    assert r["K"] == 2 and members(r) == [[0, 2], [1, 3]]
    # nodes of different GPU counts never share an island
    r = build_islands(cluster([8, 4, 8, 4], [100e12] * 4, fabric(4, 4, 1)))
    assert members(r) == [[0, 2], [1, 3]]


def test_types_interleaved_in_leaves_split_per_leaf():
    # two leaves of 2 type-A + 2 type-B nodes: A nodes of a leaf merge (their
    # 400 GB/s links tie the 400 GB/s links to the B nodes), but A nodes of two
    # leaves would have 100 GB/s inside and 400 GB/s leaving: 4 islands
    n = 8
    peak = [100e12 if u % 4 < 2 else 200e12 for u in range(n)]
    r = build_islands(cluster([8] * n, peak, fabric(n, 4, 2)))
    assert members(r) == [[0, 1], [2, 3], [4, 5], [6, 7]]


def test_types_in_separate_pods_form_one_island_each():
    n = 16
    peak = [100e12 if u < 8 else 200e12 for u in range(n)]
    r = build_islands(cluster([8] * n, peak, fabric(n, 4, 2)))
    assert members(r) == [list(range(8)), list(range(8, 16))]


def test_asymmetric_links():
    # node 2 sends to node 0 at 100 but node 0 sends to node 2 at 400: the
    # pair (0, 2) links at the slower direction; {0, 1} merges first
    e = [[0, 400e9, 400e9, 50e9], [400e9, 0, 100e9, 50e9], [100e9, 100e9, 0, 50e9], [50e9, 50e9, 50e9, 0]]
    peak = [100e12, 100e12, 100e12, 300e12]
    r = build_islands(cluster([8] * 4, peak, e))
    # {0, 1}: node 0 links 400 inside, 400 leaving (to 2): kept; then {0, 1, 2}:
    # every member's inside links >= 100 >= its links leaving (50): merged
    assert members(r) == [[0, 1, 2], [3]]
    assert r["inter_bw"] == [[0.0, 50e9], [50e9, 0.0]]


def test_island_attributes_are_sums_and_minima():
    n = 4
    peak = [100e12, 104e12, 102e12, 300e12]
    hbm = [80e9, 80e9, 80e9, 192e9]
    intra = [600e9, 590e9, 610e9, 900e9]
    host = [64e9, 32e9, 64e9, 64e9]
    e = [[0, 400e9, 400e9, 30e9], [400e9, 0, 400e9, 20e9], [400e9, 400e9, 0, 25e9], [30e9, 30e9, 30e9, 0]]
    r = build_islands(cluster([8, 8, 8, 4], peak, e, hbm=hbm, intra=intra, host=host))
    assert members(r) == [[0, 1, 2], [3]]
    isl = r["islands"]
    assert isl["n_gpus"] == [24, 4]
    assert isl["peak_flops"] == [100e12, 300e12] and isl["hbm_bytes"] == [80e9, 192e9]
    assert isl["intra_bw"] == [590e9, 900e9] and isl["host_bw"] == [32e9, 64e9]
    assert r["inter_bw"] == [[0.0, 20e9], [30e9, 0.0]]


def test_node_order_does_not_change_the_partition():
    cl = node_cluster(3, 24, n_types=3, leaf=4, pod=2, run=(2, 9))
    r = build_islands(cl)
    perm = list(np.random.default_rng(0).permutation(24))
    inv = {int(p): i for i, p in enumerate(perm)}
    nd = cl["nodes"]
    cl2 = {"nodes": {f: [nd[f][int(p)] for p in perm] for f in nd},
           "node_bw": [[cl["node_bw"][int(a)][int(b)] for b in perm] for a in perm], "eps": cl["eps"]}
    r2 = build_islands(cl2)
    part = sorted(sorted(I) for I in members(r))
    part2 = sorted(sorted(int(perm[u]) for u in I) for I in members(r2))
    assert part == part2


@pytest.mark.parametrize("bad", ["eps", "gpus", "bw"])
def test_invalid_inputs_rejected(bad):
    cl = cluster([8, 8], [1e14, 1e14], [[0, 1e11], [1e11, 0]])
    if bad == "eps":
        cl["eps"]["compute"] = -0.1
    elif bad == "gpus":
        cl["nodes"]["gpus"][0] = 0
    else:
        cl["node_bw"][0][1] = float("nan")
    with pytest.raises(OracleError) as e:
        build_islands(cl)
    assert e.value.status == EINVAL


def test_merge_order_follows_linkage_and_ties():
    # {0, 1} and {1, 2} each satisfy Eq. 3, {0, 1, 2} does not (node 0 would
    # have a 100 GB/s link inside and 300 GB/s leaving, to node 3).  Both
    # pairs link at 400 (the slower direction of 1 <-> 2 is 400, its faster
    # 450): the tie goes to the least node ids, so {0, 1} merges and 2 stays
    # alone.
    e = [[0, 400e9, 100e9, 300e9],
         [400e9, 0, 400e9, 50e9],
         [100e9, 450e9, 0, 50e9],
         [300e9, 50e9, 50e9, 0]]
    peak = [100e12, 100e12, 100e12, 400e12]  # node 3 is another GPU type
    r = build_islands(cluster([8] * 4, peak, e))
    assert members(r) == [[0, 1], [2], [3]]
