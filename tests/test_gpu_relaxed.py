"""Parity of the HIP composition with the step-(4) relaxation
(tg_compose_pipeline_relaxed, through the C ABI) with the CPU oracle's
tgo_compose_relaxed: the plan (b, stages, islands, cuts, configs, pair
indices, bound P, F, T and per-stage values) compared bit for bit.  Cases
include instances where relaxing the bound changes the plan and the chosen b,
random tiny instances (the seeds where it pays and others), and the
128-island instance against the oracle's stored result."""
import copy
import sys

import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from oracle.oracle import Oracle  # noqa: E402
from workloads import load_instance, random_tiny  # noqa: E402
from tests.inst_util import instance, tiny_tight  # noqa: E402
from tests.golden.make_golden import load as load_golden  # noqa: E402
from tests.test_gpu_parity import plan_equal  # noqa: E402

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2606_16907_amd import tangram as T  # noqa: E402

# random tiny instances where the relaxed plan beats steps (1)-(3), plus others
IMPROVING = [4, 10, 13, 15, 21, 41, 52, 68, 72, 100, 104, 114, 119]
OTHERS = [0, 1, 2, 3, 5, 6, 7, 8]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _batch(name, B):
    def make():
        inst = copy.deepcopy(load_instance(name))
        inst["space"]["global_batch"] = B
        inst["name"] = f"{name}_B{B}"
        return inst
    return make


def _two_island():
    return instance(L=2, K=2, layer={"fwd_flops": 2 ** 40, "out_act_bytes": 3 * 2 ** 29},
                    peak=3.0 * 2 ** 40, hbm=2.0 ** 60, inter=2.0 ** 31, B=2)


CASES = ([("two_island", _two_island), ("tiny", lambda: load_instance("tiny")), ("tiny_tight", tiny_tight),
          ("dense8b", lambda: load_instance("dense8b")), ("moe_B64", _batch("moe", 64)),
          ("moe_B128", _batch("moe", 128)), ("dense70b_B64", _batch("dense70b", 64))]
         + [(f"rand{s}", lambda s=s: random_tiny(s, tight=(s % 2 == 1))) for s in IMPROVING + OTHERS])


def _gpu_relaxed(p):
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    st, plan = p.tg_compose_pipeline_relaxed(surv, cost, dmax)
    st3, plan3 = p.tg_compose_pipeline(surv, cost, dmax)
    return st, plan, st3, plan3


@pytest.mark.parametrize("name,make", CASES, ids=[n for n, _ in CASES])
def test_relaxed_parity(name, make):
    inst = make()
    say("case", name)
    o = Oracle(inst)
    s = o.prune()
    ost, oplan, _ = o.compose_relaxed(s)
    p = T.Problem(inst)
    st, plan, st3, plan3 = _gpu_relaxed(p)
    if ost != 0:
        assert st == T.TG_ENOPLAN and plan["S"] == 0
        return
    assert st == 0
    plan_equal(plan, oplan)
    # never worse than steps (1)-(3), which stay unchanged by the relaxed call
    o3 = o.compose(s)[1]
    plan_equal(plan3, o3)
    assert plan["T"] <= plan3["T"]


def test_relaxed_changes_the_plan_where_it_pays():
    o = Oracle(_batch("moe", 64)())
    s = o.prune()
    a = o.compose(s)[1]
    b = o.compose_relaxed(s)[1]
    assert b["T"] < a["T"] and b["b"] != a["b"]
    p = T.Problem(o.inst)
    st, plan, st3, plan3 = _gpu_relaxed(p)
    assert plan["b"] == b["b"] and plan["T"] == b["T"] and plan3["T"] == a["T"]


def test_relaxed_large_instance_against_stored_oracle_result():
    g = load_golden("large")
    inst = load_instance("large")
    say("case large relaxed")
    p = T.Problem(inst)
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    assert int(surv.numel()) == g["survivors"]["count"]
    st, plan = p.tg_compose_pipeline_relaxed(surv, cost, dmax)
    assert st == 0
    plan_equal(plan, g["relaxed"]["plan"])


def test_relaxed_workspace_and_arguments():
    inst = load_instance("tiny")
    p = T.Problem(inst)
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    lib = T.load_library()
    assert lib.tg_compose_relaxed_workspace_bytes(p.h, int(surv.numel())) >= \
        lib.tg_compose_workspace_bytes(p.h, int(surv.numel()))
    small = p.compose_workspace(int(surv.numel()))  # too small for the relaxed search
    with pytest.raises(T.TangramError):
        p.tg_compose_pipeline_relaxed(surv, cost, dmax, workspace=small[:16])
    with pytest.raises(T.TangramError):
        p.tg_compose_pipeline_relaxed(surv, cost, dmax, island_order=[0, 0])
    st, plan = p.tg_compose_pipeline_relaxed(surv[:0], cost, dmax)
    assert st == T.TG_ENOPLAN and plan["S"] == 0
