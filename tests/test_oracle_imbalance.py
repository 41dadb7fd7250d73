"""Pins of the oracle's imbalance pruning (Sec. 5.1 (ii)): a model-slice /
island pair is dropped when the slice's share of the model's forward FLOPs
and the island's share of the cluster's compute (GPUs x peak FLOP/s) are
mismatched by more than a factor 1 + eps either way (over-subscription stalls
the island, under-subscription leaves it idle).  The paper gives no tolerance;
eps is an input, 0 = off.  Checked by closed forms on power-of-two shares,
invariants in eps, and exhaustive composition over the kept pairs."""
import copy
import math

import numpy as np
import pytest

from oracle.oracle import Oracle, OracleError, EINVAL, ENOPLAN
from workloads import random_tiny
from tests import brute
from tests.inst_util import instance


def with_eps(inst, eps):
    out = copy.deepcopy(inst)
    out["space"]["imbalance_eps"] = float(eps)
    return out


def _random(seed, eps):
    return with_eps(random_tiny(seed, tight=(seed % 2 == 1)), eps)


def test_closed_form_two_islands():
    # island 0: 3 GPUs, island 1: 1 GPU of the same peak -> shares 3/4, 1/4.
    # 8 equal layers: slice [i, j) demands (j - i) / 8.  eps = 1/2:
    #   island 0 keeps 3/4 / (3/2) <= q <= 3/4 * 3/2, i.e. 4..8 layers;
    #   island 1 keeps 1/4 / (3/2) <= q <= 1/4 * 3/2, i.e. 2..3 layers.
    inst = instance(K=2, L=8, layer={"fwd_flops": 2 ** 40}, n_gpus=[3, 1], B=4, tp=(1,), mb=(1,), zero=(0,))
    o = Oracle(with_eps(inst, 0.5))
    keep = {0: range(4, 9), 1: range(2, 4)}
    for i in range(8):
        for j in range(i + 1, 9):
            for k in (0, 1):
                assert o.balanced(i, j, k) == ((j - i) in keep[k]), (i, j, k)
    got = {(o.decode(x)["i"], o.decode(x)["j"], o.decode(x)["island"]) for x in o.prune()}
    for (i, j, k) in got:
        assert (j - i) in keep[k]


def test_zero_eps_is_off_and_huge_eps_keeps_every_pair():
    for seed in range(12):
        base = Oracle(_random(seed, 0.0)).prune().tolist()
        assert base == Oracle(random_tiny(seed, tight=(seed % 2 == 1))).prune().tolist()
        assert base == Oracle(_random(seed, 1e12)).prune().tolist()


@pytest.mark.parametrize("seed", range(16))
def test_survivors_shrink_as_eps_shrinks(seed):
    prev = None
    for eps in (4.0, 1.0, 0.5, 0.25, 0.125):
        s = set(Oracle(_random(seed, eps)).prune().tolist())
        if prev is not None:
            assert s <= prev
        prev = s


@pytest.mark.parametrize("seed", range(16))
def test_kept_pairs_are_the_dominance_survivors_of_balanced_groups(seed):
    o = Oracle(_random(seed, 0.5))
    off = Oracle(random_tiny(seed, tight=(seed % 2 == 1)))
    want = [x for x in off.prune().tolist()
            if o.balanced(off.decode(x)["i"], off.decode(x)["j"], off.decode(x)["island"])]
    assert o.prune().tolist() == want


def _allowed(o):
    B = o.inst["space"]["global_batch"]
    out = set()
    for idx in range(o.N):
        t = o.decode(idx)
        if B % (t["dp"] * t["mb"]) == 0 and o.balanced(t["i"], t["j"], t["island"]):
            out.add(idx)
    return out


@pytest.mark.parametrize("seed", range(40))
def test_compositions_equal_exhaustive_search_over_kept_pairs(seed):
    eps = (0.25, 0.5, 1.0)[seed % 3]
    o = Oracle(_random(seed, eps))
    rows = brute.candidate_table(o)
    allowed = _allowed(o)
    s = o.prune()
    st, plan, per_b = o.compose(s)
    bf, best = brute.brute_force_compose(o, rows, allowed=allowed)
    if best is None:
        assert st == ENOPLAN
    else:
        assert (plan["b"], plan["P"], plan["F"], plan["T"]) == (best["b"], best["P"], best["F"], best["T"])
        for x in plan["stages"]:
            assert o.balanced(x["first_layer"], x["end_layer"], x["island"])
    st, plan, _ = o.compose_relaxed(s)
    bf, best = brute.brute_force_relaxed(o, rows, allowed=allowed)
    if best is not None:
        assert (plan["b"], plan["P"], plan["F"], plan["T"]) == (best["b"], best["P"], best["F"], best["T"])
    st, plan, _ = o.compose_all_orders(s)
    bf, best = brute.brute_force_all_orders(o, rows, allowed=allowed)
    if best is None:
        assert st == ENOPLAN
    else:
        assert (plan["b"], plan["P"], plan["F"], plan["T"]) == (best["b"], best["P"], best["F"], best["T"])


def test_compose_rejects_unbalanced_pairs():
    inst = instance(K=2, L=8, layer={"fwd_flops": 2 ** 40}, n_gpus=[3, 1], B=4, tp=(1,), mb=(1,), zero=(0,))
    o = Oracle(with_eps(inst, 0.5))
    # slice [0, 1) on island 0 (one layer, demand 1/8 against share 3/4) is unbalanced
    assert not o.balanced(0, 1, 0)
    assert o.compose([0])[0] == EINVAL
    assert o.compose_all_orders([0])[0] == EINVAL


@pytest.mark.parametrize("bad", [-0.5, float("nan"), float("inf")])
def test_invalid_eps_rejected(bad):
    with pytest.raises(OracleError) as e:
        Oracle(with_eps(random_tiny(0), bad))
    assert e.value.status == EINVAL


def test_model_without_flops_is_never_pruned():
    inst = instance(K=2, L=3, layer={"act_stash_bytes": 2 ** 20}, n_gpus=[3, 1], B=2)
    assert Oracle(with_eps(inst, 0.1)).prune().tolist() == Oracle(inst).prune().tolist()
