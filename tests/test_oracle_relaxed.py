"""Pins of the oracle's composition with the relaxation of step (4) (Sec. 5.2):
the bottleneck bound is raised over the stage and link costs above P* until
the iteration time T = (m-1) * P + F stops improving.  The exact result is the
least T over every plan, which exhaustive search computes directly."""
import math

import numpy as np
import pytest

from oracle.oracle import Oracle, ENOPLAN
from workloads import make_instance, random_tiny
from tests import brute
from tests.inst_util import instance, tiny_tight
from tests.test_oracle_search import check_plan_invariants

RANDOM_SEEDS = list(range(120))


def _random(seed):
    return random_tiny(seed, tight=(seed % 2 == 1))


def _check_relaxed(o, rows, order=None):
    surv = o.prune()
    st, plan, per_b = o.compose_relaxed(surv, order)
    bf_per_b, best = brute.brute_force_relaxed(o, rows, order)
    for bi, b in enumerate(o.bvalues):
        want = bf_per_b[b]
        if math.isinf(want[0]):
            assert math.isinf(per_b[bi][0])
        else:
            assert tuple(per_b[bi]) == want, (b, per_b[bi], want)
    if best is None:
        assert st == ENOPLAN
        return None
    assert st == 0
    assert (plan["b"], plan["P"], plan["F"], plan["T"]) == (best["b"], best["P"], best["F"], best["T"])
    order = order if order is not None else o.inst["island_order"]
    sig = brute.plan_signature(plan)
    optimal = {brute.brute_signature(p, order): p for p in best["optimal"]}
    assert sig in optimal, "oracle plan is not among the optimal plans"
    lex = brute.brute_signature(best["lexmin"], order)
    if sig != lex:
        # ties broken differently only through floating-point absorption
        mine, other = optimal[sig], best["lexmin"]
        t = next(t for t in range(min(len(sig), len(lex))) if sig[t] != lex[t])
        assert brute.suffix_values(mine)[t] != brute.suffix_values(other)[t]
    return plan


def test_relaxed_equals_exhaustive_search_on_random_instances():
    improved = 0
    for seed in RANDOM_SEEDS:
        o = Oracle(_random(seed))
        rows = brute.candidate_table(o)
        plan = _check_relaxed(o, rows)
        if plan is not None:
            st, base, _ = o.compose(o.prune())
            assert plan["T"] <= base["T"]
            improved += plan["T"] < base["T"]
    # the seeds include instances where relaxing the bound pays
    assert improved >= 1


def test_relaxed_exhaustive_tiny_and_tight():
    for inst in (make_instance("tiny"), tiny_tight()):
        o = Oracle(inst)
        _check_relaxed(o, brute.candidate_table(o))


def test_relaxed_with_other_orders():
    o = Oracle(random_tiny(3, L_range=(5, 5), K_range=(3, 3)))
    rows = brute.candidate_table(o)
    for order in ([0, 1, 2], [2, 1, 0], [1, 0, 2]):
        _check_relaxed(o, rows, order)


def _two_island_instance(B):
    # one layer costs exactly 1 s on either island (3 * 2^40 FLOP at 3 * 2^40
    # FLOP/s, a single GPU, no communication terms); the link carries
    # 2 * b * 3 * 2^29 bytes at 2^31 B/s = 1.5 s for b = 1
    return instance(L=2, K=2, layer={"fwd_flops": 2 ** 40, "out_act_bytes": 3 * 2 ** 29},
                    peak=3.0 * 2 ** 40, hbm=2.0 ** 60, inter=2.0 ** 31, B=B)


def test_relaxation_closed_form():
    # Two plans exist: split (1 layer per island, P = 1.5 the link, F = 1 +
    # (1.5 + 1) = 3.5) and whole (both layers on one island, P = F = 2).  With
    # m = 2: steps (1)-(3) take the split at P* = 1.5, T = 1.5 + 3.5 = 5; the
    # relaxed bound 2 admits the whole plan, T = 2 + 2 = 4.
    o = Oracle(_two_island_instance(B=2))
    s = o.prune()
    st, base, per3 = o.compose(s)
    assert st == 0 and (base["P"], base["F"], base["T"], base["S"]) == (1.5, 3.5, 5.0, 2)
    st, plan, per4 = o.compose_relaxed(s)
    assert st == 0 and (plan["P"], plan["F"], plan["T"], plan["S"]) == (2.0, 2.0, 4.0, 1)
    assert plan["stages"][0]["island"] == 0
    assert tuple(per4[0]) == (1.5, 2.0, 2.0, 4.0)
    check_plan_invariants(o, plan, s)


def test_single_microbatch_minimises_fill():
    # m = 1: T = F, so the relaxed plan is the least-fill plan over all bounds
    o = Oracle(_two_island_instance(B=1))
    s = o.prune()
    st, plan, _ = o.compose_relaxed(s)
    assert st == 0 and plan["m"] == 1 and (plan["T"], plan["F"], plan["P"]) == (2.0, 2.0, 2.0)
    rows = brute.candidate_table(o)
    plans = brute.enumerate_plans(o, rows)[1]
    assert plan["T"] == min(p["F"] for p in plans)


def test_no_improvement_keeps_step3_plan():
    # with a fast link (x = 0.5 s) the split plan has both the least P and the
    # least T, so the relaxed search returns exactly the steps-(1)-(3) plan
    inst = _two_island_instance(B=2)
    inst["inter_bw"] = [[0.0, 2.0 ** 33], [2.0 ** 33, 0.0]]
    o = Oracle(inst)
    s = o.prune()
    a = o.compose(s)
    b = o.compose_relaxed(s)
    assert a[1] == b[1]
    assert (b[1]["P"], b[1]["T"]) == (1.0, 1.0 + (1.0 + (0.375 + 1.0)))


@pytest.mark.parametrize("name", ["tiny", "dense8b", "moe"])
def test_relaxed_named_instances(name):
    o = Oracle(make_instance(name))
    s = o.prune()
    st3, p3, per3 = o.compose(s)
    st, plan, per = o.compose_relaxed(s)
    assert st == 0
    check_plan_invariants(o, plan, s)
    assert plan["T"] == min(per[:, 3]) <= p3["T"]
    # P* is the same; per b the relaxed T never exceeds the steps-(1)-(3) T
    fin = np.isfinite(per3[:, 0])
    assert np.array_equal(per[fin, 0], per3[fin, 0])
    assert np.all(per[fin, 3] <= per3[fin, 2])
    assert np.all(per[fin, 1] >= per[fin, 0])


def test_relaxed_infeasible_instance():
    from tests.inst_util import scaled
    inst = scaled(make_instance("tiny"), memory=1e-6)
    o = Oracle(inst)
    st, plan, _ = o.compose_relaxed(o.prune())
    assert st == ENOPLAN and plan["S"] == 0 and math.isinf(plan["T"])
