"""Pins of the oracle's redundancy pruning (Sec. 5.1 (i)): slices of the same
composition are one query.  Two slices are equivalent when all their
per-slice sums are equal; every config then scores them alike, so the
surviving set found once per class and copied to the class's slices is the
surviving set itself.  Checked against the definition (brute-force classes,
per-candidate scores), closed forms (uniform and repeating layers), and the
plain surviving set (random, tight, imbalance-pruned and extended
instances, the named small instances)."""
import copy

import numpy as np
import pytest

from oracle.oracle import Oracle
from workloads import extended, make_instance, random_tiny
from tests.inst_util import instance

SUMS = ("fwd_flops", "dense_params", "expert_params", "act_stash_bytes", "tp_comm_bytes", "a2a_bytes",
        "out_act_bytes", "cp_comm_bytes")


def slices(L):
    return [(i, j) for i in range(L) for j in range(i + 1, L + 1)]


def sum_vector(inst, i, j):
    lay = inst["layers"]
    return tuple(sum(lay.get(f, [0] * len(lay["fwd_flops"]))[i:j]) for f in SUMS)


def _random(seed):
    inst = random_tiny(seed, tight=(seed % 2 == 1))
    if seed % 4 == 0:  # repeat the first two layers: equal compositions appear
        for f in inst["layers"]:
            v = inst["layers"][f]
            inst["layers"][f] = (v[:2] * (len(v) // 2 + 1))[:len(v)]
    return inst


@pytest.mark.parametrize("seed", range(16))
def test_classes_are_equal_sum_vectors(seed):
    inst = _random(seed)
    o = Oracle(inst)
    cls, nc = o.slice_classes()
    sl = slices(o.L)
    vec = [sum_vector(inst, i, j) for i, j in sl]
    for a in range(len(sl)):
        for b in range(len(sl)):
            assert (cls[a] == cls[b]) == (vec[a] == vec[b])
    # numbered in the order of first slices
    firsts = [list(cls).index(c) for c in range(nc)]
    assert firsts == sorted(firsts) and nc == len(set(vec))


def test_uniform_layers_are_one_class_per_length():
    inst = instance(L=7, K=2, layer={"fwd_flops": 2 ** 40, "dense_params": 2 ** 20, "act_stash_bytes": 2 ** 20})
    o = Oracle(inst)
    cls, nc = o.slice_classes()
    sl = slices(7)
    assert nc == 7
    for a, (i, j) in enumerate(sl):
        for b, (i2, j2) in enumerate(sl):
            assert (cls[a] == cls[b]) == (j - i == j2 - i2)


def test_repeating_pair_of_layers():
    # layers A B A B A B: a slice's class is its length and, for odd lengths,
    # whether it starts on A
    lay = {"fwd_flops": [2 ** 40, 3 * 2 ** 38] * 3, "dense_params": [2 ** 20, 2 ** 21] * 3}
    o = Oracle(instance(K=1, layers=lay))
    cls, nc = o.slice_classes()
    key = {}
    for a, (i, j) in enumerate(slices(6)):
        k = (j - i, i % 2 if (j - i) % 2 else 0)
        key.setdefault(k, set()).add(int(cls[a]))
    assert all(len(v) == 1 for v in key.values()) and nc == len(key) == 9


@pytest.mark.parametrize("seed", range(8))
def test_equivalent_slices_score_alike(seed):
    o = Oracle(_random(seed))
    cls, nc = o.slice_classes()
    cost, dmax = o.score()
    first = {int(c): s for s, c in reversed(list(enumerate(cls)))}
    for g in range(o.n_configs):
        for s in range(o.NS):
            r = first[int(cls[s])]
            assert cost[g * o.NS + s] == cost[g * o.NS + r] and dmax[g * o.NS + s] == dmax[g * o.NS + r]


@pytest.mark.parametrize("seed", range(24))
def test_redundancy_pruned_set_is_the_surviving_set(seed):
    inst = _random(seed)
    if seed % 3 == 1:
        inst = copy.deepcopy(inst)
        inst["space"]["imbalance_eps"] = 0.5
    if seed % 5 == 2:
        inst = extended(inst, cp=(1, 2), recompute=(0, 1), offload=(0, 1))
    o = Oracle(inst)
    assert np.array_equal(o.prune_classes(), o.prune())


@pytest.mark.parametrize("name", ["tiny", "dense8b"])
def test_named_instances(name):
    o = Oracle(make_instance(name))
    cls, nc = o.slice_classes()
    assert nc == o.L  # uniform decoder layers: one class per slice length
    assert np.array_equal(o.prune_classes(), o.prune())


def test_slices_differing_only_in_later_sums_are_different_classes():
    # layers A B A B: A and B agree on FLOPs, parameters and stash and differ
    # only in output activation and key/value bytes
    lay = {"fwd_flops": [2 ** 40] * 4, "dense_params": [2 ** 20] * 4, "act_stash_bytes": [2 ** 20] * 4,
           "out_act_bytes": [2 ** 10, 2 ** 11, 2 ** 10, 2 ** 11], "cp_comm_bytes": [3, 5, 3, 5]}
    o = Oracle(instance(K=1, layers=lay))
    cls, nc = o.slice_classes()
    idx = {sl: a for a, sl in enumerate(slices(4))}
    assert cls[idx[(0, 1)]] == cls[idx[(2, 3)]] != cls[idx[(1, 2)]] == cls[idx[(3, 4)]]
    assert cls[idx[(0, 2)]] == cls[idx[(1, 3)]] == cls[idx[(2, 4)]]
    assert nc == 6  # length 1: A, B; 2: AB = BA; 3: ABA, BAB; 4
