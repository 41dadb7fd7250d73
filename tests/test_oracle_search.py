"""Pins of the oracle's pruning and composition against exhaustive search,
textbook reductions and the behaviours the paper reports (Sec. 5.1, 5.2, 6)."""
import math

import numpy as np
import pytest

from oracle.oracle import Oracle, ENOPLAN, EINVAL
from workloads import make_instance, random_tiny
from tests import brute
from tests.inst_util import instance, scaled, tiny_tight

RANDOM_SEEDS = list(range(120))


def _random(seed):
    return random_tiny(seed, tight=(seed % 2 == 1))


# ---------------------------------------------------------------------------
# surviving set
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(40))
def test_survivors_match_both_definitions(seed):
    o = Oracle(_random(seed))
    rows = brute.candidate_table(o)
    got = o.prune().tolist()
    assert got == brute.survivors_by_reps(rows, o.K)
    assert got == brute.survivors_by_dominance(rows)


def test_survivors_tiny_and_tight():
    for inst in (make_instance("tiny"), tiny_tight()):
        o = Oracle(inst)
        rows = brute.candidate_table(o)
        assert o.prune().tolist() == brute.survivors_by_reps(rows, o.K)


# ---------------------------------------------------------------------------
# composition vs exhaustive search over every plan
# ---------------------------------------------------------------------------
def _check_against_brute(o, rows, order=None):
    surv = o.prune()
    st, plan, per_b = o.compose(surv, order)
    bf_per_b, best = brute.brute_force_compose(o, rows, order)
    for bi, b in enumerate(o.bvalues):
        P, F, T = bf_per_b[b]
        if math.isinf(P):
            assert math.isinf(per_b[bi][0])
        else:
            assert tuple(per_b[bi]) == (P, F, T), (b, per_b[bi], (P, F, T))
    if best is None:
        assert st == ENOPLAN
        return "noplan"
    assert st == 0
    assert (plan["b"], plan["P"], plan["F"], plan["T"]) == (best["b"], best["P"], best["F"], best["T"])
    order = order if order is not None else o.inst["island_order"]
    sig = brute.plan_signature(plan)
    optimal = {brute.brute_signature(p, order): p for p in best["optimal"]}
    assert sig in optimal, "oracle plan is not among the optimal plans"
    lex = brute.brute_signature(best["lexmin"], order)
    if sig == lex:
        return "lexmin"
    # Differs only through floating-point absorption: at the first stage where
    # the two plans part, their suffix fills differ although both totals tie.
    mine, other = optimal[sig], best["lexmin"]
    t = next(t for t in range(min(len(sig), len(lex))) if sig[t] != lex[t])
    assert brute.suffix_values(mine)[t] != brute.suffix_values(other)[t]
    return "absorbed"


@pytest.mark.parametrize("seed", RANDOM_SEEDS)
def test_compose_equals_exhaustive_search(seed):
    o = Oracle(_random(seed))
    rows = brute.candidate_table(o)
    _check_against_brute(o, rows)


def test_compose_exhaustive_tiny_and_tight():
    outcomes = []
    for inst in (make_instance("tiny"), tiny_tight()):
        o = Oracle(inst)
        outcomes.append(_check_against_brute(o, brute.candidate_table(o)))
    assert outcomes[0] == "lexmin"


def test_compose_exhaustive_with_other_orders():
    o = Oracle(random_tiny(3, L_range=(5, 5), K_range=(3, 3)))
    rows = brute.candidate_table(o)
    for order in ([0, 1, 2], [2, 1, 0], [1, 0, 2]):
        _check_against_brute(o, rows, order)


# ---------------------------------------------------------------------------
# dominance pruning never changes the composed plan
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(30))
def test_prune_safety(seed):
    o = Oracle(_random(seed))
    cost, dmax = o.score()
    B = o.inst["space"]["global_batch"]
    compatible = [i for i in range(o.N)
                  if B % (o.decode(i)["dp"] * o.decode(i)["mb"]) == 0]
    a = o.compose(o.prune())
    b = o.compose(compatible)
    assert a[0] == b[0]
    assert a[1] == b[1]
    assert np.array_equal(a[2], b[2])


def test_prune_safety_dense8b():
    o = Oracle(make_instance("dense8b"))
    cost, dmax = o.score()
    B = o.inst["space"]["global_batch"]
    ok = []
    for g in range(o.n_configs):
        t = o.decode(g * o.NS)
        if B % (t["dp"] * t["mb"]) == 0:
            ok.append(np.arange(g * o.NS, (g + 1) * o.NS))
    allc = np.concatenate(ok)
    allc = allc[dmax[allc] >= 1]
    a = o.compose(o.prune())
    b = o.compose(allc)
    assert a[1] == b[1] and np.array_equal(a[2], b[2])


def test_compose_rejects_incompatible_and_unsorted():
    o = Oracle(make_instance("tiny"))
    B = o.inst["space"]["global_batch"]
    bad = next(i for i in range(o.N) if B % (o.decode(i)["dp"] * o.decode(i)["mb"]) != 0)
    assert o.compose([bad])[0] == EINVAL
    s = o.prune()
    assert o.compose(s[::-1])[0] == EINVAL
    assert o.compose(s, order=[0, 0])[0] == EINVAL


# ---------------------------------------------------------------------------
# textbook reductions
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(8))
def test_reduces_to_linear_partition(seed):
    # identical islands, unbounded memory, free links, one config: the least
    # bottleneck is the classic min-max contiguous partition of the layer
    # FLOPs into at most K parts, scaled by 3/F (exact: F = 3 * 2^40)
    rng = np.random.default_rng(100 + seed)
    L = int(rng.integers(3, 14))
    K = int(rng.integers(1, 6))
    flops = [int(x) for x in rng.integers(1, 1000, size=L)]
    inst = instance(L=L, K=K, layers={"fwd_flops": flops}, peak=3.0 * 2.0 ** 40,
                    hbm=2.0 ** 60, inter=math.inf, B=1)
    o = Oracle(inst)
    st, plan, per_b = o.compose(o.prune())
    assert st == 0
    assert plan["P"] == brute.linear_partition_minmax(flops, K) * 2.0 ** -40


@pytest.mark.parametrize("L,K", [(8, 3), (8, 8), (8, 12), (5, 2), (16, 5)])
def test_uniform_layers_closed_form(L, K):
    # uniform layers on identical islands with free links: the bottleneck is
    # the cost of ceil(L / min(K, L)) layers
    inst = instance(L=L, K=K, layer={"fwd_flops": 2 ** 40}, peak=3.0 * 2.0 ** 40,
                    hbm=2.0 ** 60, inter=math.inf, B=1)
    o = Oracle(inst)
    st, plan, _ = o.compose(o.prune())
    assert plan["P"] == float(-(-L // min(K, L)))


def test_transfer_term_closed_form():
    # two 1-layer islands that can only hold one layer each: the link after
    # layer 0 carries 2 * b * out_act bytes at E bytes/s
    inst = instance(L=2, K=2, layer={"fwd_flops": 2 ** 40, "dense_params": 2 ** 20,
                                     "out_act_bytes": 2 ** 30},
                    peak=3.0 * 2.0 ** 40, hbm=16.0 * 2 ** 20 * 1.5, inter=2.0 ** 31, B=2,
                    mb=(1, 2))
    o = Oracle(inst)
    st, plan, _ = o.compose(o.prune())
    assert st == 0 and plan["S"] == 2
    b = plan["b"]
    assert plan["stages"][0]["link_out"] == 2.0 * b * 2 ** 30 / 2 ** 31
    assert plan["P"] == max(s["cost"] for s in plan["stages"] + [{"cost": plan["stages"][0]["link_out"]}])


# ---------------------------------------------------------------------------
# behaviours reported in the paper
# ---------------------------------------------------------------------------
def test_single_island_runs_whole_model():
    # one island: one model slice holding the whole model (Sec. 6.6)
    inst = make_instance("tiny")
    inst = dict(inst, islands={k: v[:1] for k, v in inst["islands"].items()},
                inter_bw=[[0.0]], island_order=[0])
    o = Oracle(inst)
    st, plan, _ = o.compose(o.prune())
    assert st == 0 and plan["S"] == 1
    assert (plan["stages"][0]["first_layer"], plan["stages"][0]["end_layer"]) == (0, o.L)


def test_slow_island_is_eliminated():
    # a resource-limited island that would bottleneck the pipeline is left out
    # (Sec. 5.2 island elimination; Sec. 6.4 configuration (iii))
    base = make_instance("dense8b")
    o = Oracle(base)
    st, plan, _ = o.compose(o.prune())
    used = {s["island"] for s in plan["stages"]}
    slow = base["island_order"][0]
    assert slow in used
    inst = scaled(base)
    inst["islands"]["peak_flops"][slow] = 1e9   # a thousand times slower than any GPU
    o2 = Oracle(inst)
    st2, plan2, _ = o2.compose(o2.prune())
    assert st2 == 0 and slow not in {s["island"] for s in plan2["stages"]}


def test_order_matters_under_memory_pressure():
    # memory-rich islands first vs last gives different pipelines when memory
    # binds (the Sec. 6.2 observation that a different island order changes the
    # iteration time)
    # island 0: slow, 16 GiB; island 1: 4x faster, 3 GiB.  Each layer stashes
    # 1 GiB per micro-batch, so the small island holds two layers at the end of
    # the pipeline (depth 1) but only one layer at its front (depth 2).
    inst = instance(L=4, K=2, layer={"fwd_flops": 2 ** 40, "dense_params": 2 ** 10,
                                     "act_stash_bytes": 2 ** 30},
                    peak=[3.0 * 2 ** 40, 12.0 * 2 ** 40], hbm=[16.0 * 2 ** 30, 3.0 * 2 ** 30],
                    inter=math.inf, B=8)
    o = Oracle(inst)
    s = o.prune()
    st_a, a, _ = o.compose(s, [0, 1])
    st_b, b, _ = o.compose(s, [1, 0])
    assert st_a == st_b == 0
    assert a["P"] == 2.0 and b["P"] == 3.0
    assert [(x["island"], x["end_layer"] - x["first_layer"]) for x in a["stages"]] == [(0, 2), (1, 2)]
    assert [(x["island"], x["end_layer"] - x["first_layer"]) for x in b["stages"]] == [(1, 1), (0, 3)]


def test_infeasible_instance_has_no_plan():
    inst = scaled(make_instance("tiny"), memory=1e-6)
    o = Oracle(inst)
    s = o.prune()
    assert len(s) == 0
    st, plan, _ = o.compose(s)
    assert st == ENOPLAN and plan["S"] == 0 and math.isinf(plan["T"])


# ---------------------------------------------------------------------------
# invariants of the plans on the named instances
# ---------------------------------------------------------------------------
def check_plan_invariants(o, plan, survivors):
    inst = o.inst
    B = inst["space"]["global_batch"]
    st = plan["stages"]
    assert plan["S"] == len(st) >= 1
    assert B % plan["b"] == 0 and plan["m"] == B // plan["b"]
    assert st[0]["first_layer"] == 0 and st[-1]["end_layer"] == o.L
    for a, c in zip(st, st[1:]):
        assert a["end_layer"] == c["first_layer"]
    assert all(s["first_layer"] < s["end_layer"] for s in st)
    islands = [s["island"] for s in st]
    assert len(set(islands)) == len(islands)
    pos = {k: p for p, k in enumerate(inst["island_order"])}
    assert [pos[k] for k in islands] == sorted(pos[k] for k in islands)
    surv = set(int(x) for x in survivors)
    costs, dms = o.score_list([s["pair_index"] for s in st])
    for t, s in enumerate(st):
        assert s["depth"] == plan["S"] - t
        assert s["pair_index"] in surv
        d = o.decode(s["pair_index"])
        assert (d["i"], d["j"], d["island"]) == (s["first_layer"], s["end_layer"], s["island"])
        assert (d["tp"], d["dp"], d["ep"], d["zero"], d["mb"]) == \
            (s["tp"], s["dp"], s["ep"], s["zero"], s["mb"])
        assert s["dp"] * s["mb"] == plan["b"]
        assert s["tp"] * s["dp"] <= inst["islands"]["n_gpus"][s["island"]]
        assert costs[t] == s["cost"] and dms[t] >= s["depth"]
        assert s["mem_bytes"] <= inst["islands"]["hbm_bytes"][s["island"]] * inst["space"]["mem_frac"]
    f = [s["cost"] for s in st]
    x = [s["link_out"] for s in st[:-1]]
    assert plan["P"] == max(f + x)
    assert plan["F"] == brute.right_fold(f, x)
    assert plan["T"] == (float(plan["m"] - 1) * plan["P"]) + plan["F"]


@pytest.mark.parametrize("name", ["tiny", "dense8b", "dense70b", "moe"])
def test_named_instance_plan_invariants(name):
    o = Oracle(make_instance(name))
    s = o.prune()
    st, plan, per_b = o.compose(s)
    assert st == 0
    check_plan_invariants(o, plan, s)
    assert plan["T"] == min(per_b[:, 2])


def test_oracle_refuses_plans_whose_m_overflows_int32():
    """The plan reports m = B / b as a 32-bit integer: B = 2^31 with b = 1
    compatible is refused at create."""
    from oracle.oracle import OracleError
    from tests.inst_util import instance
    with pytest.raises(OracleError) as e:
        Oracle(instance(L=2, K=1, layer={"fwd_flops": 2**30}, B=2**31))
    assert e.value.status == EINVAL
    Oracle(instance(L=2, K=1, layer={"fwd_flops": 2**30}, B=2**31 - 1))
