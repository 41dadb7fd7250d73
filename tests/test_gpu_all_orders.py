"""Parity of the HIP composition over every island subset and order
(tg_compose_pipeline_all_orders, through the C ABI) with the CPU oracle's
tgo_compose_all_orders: the plan (b, stages, islands, cuts, configs, pair
indices, P, F, T and per-stage values) compared bit for bit.  Cases: the
named instances with at most 16 islands (the 16-island 70B instance against
the oracle's stored result), random instances from one to eight islands,
instances with exact ties, models longer than one block of threads, fewer
layers than islands, the extended config space, an empty list and the
16-island limit."""
import ctypes
import sys

import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from oracle.oracle import Oracle  # noqa: E402
from workloads import extended, load_instance, random_tiny  # noqa: E402
from tests.inst_util import scaled, tiny_tight  # noqa: E402
from tests.golden.make_golden import load as load_golden  # noqa: E402
from tests.test_gpu_parity import plan_equal  # noqa: E402
from tests.test_oracle_all_orders import _symmetric  # noqa: E402

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2606_16907_amd import tangram as T  # noqa: E402


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


CASES = ([("tiny", lambda: load_instance("tiny")), ("tiny_tight", tiny_tight),
          ("dense8b", lambda: load_instance("dense8b")),
          ("dense8b_ext", lambda: extended(load_instance("dense8b")))]
         + [(f"rand{s}", lambda s=s: random_tiny(s, tight=(s % 2 == 1))) for s in range(16)]
         + [(f"sym{s}", lambda s=s: _symmetric(s)) for s in range(8)]
         + [(f"wide{s}", lambda s=s: random_tiny(2000 + s, L_range=(6, 12), K_range=(5, 8), tight=(s % 2 == 1)))
            for s in range(6)]
         + [("long70", lambda: random_tiny(3000, L_range=(70, 70), K_range=(3, 3))),
            ("long140", lambda: random_tiny(3001, L_range=(140, 140), K_range=(2, 2), tight=True)),
            ("long300", lambda: scaled(random_tiny(3006, L_range=(300, 300), K_range=(3, 3)), memory=64.0)),
            ("few_layers", lambda: random_tiny(3002, L_range=(2, 3), K_range=(5, 6))),
            ("one_island", lambda: random_tiny(3003, L_range=(5, 5), K_range=(1, 1)))])


def _gpu(p):
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    return surv, cost, dmax


@pytest.mark.parametrize("name,make", CASES, ids=[n for n, _ in CASES])
def test_all_orders_parity(name, make):
    inst = make()
    say("case", name)
    o = Oracle(inst)
    ost, oplan, _ = o.compose_all_orders(o.prune())
    p = T.Problem(inst)
    surv, cost, dmax = _gpu(p)
    ws = p.compose_all_orders_workspace(int(surv.numel()))
    for rep in range(2):  # the same workspace twice: nothing carries over
        st, plan = p.tg_compose_pipeline_all_orders(surv, cost, dmax, workspace=ws)
        if ost != 0:
            assert st == T.TG_ENOPLAN and plan["S"] == 0
            continue
        assert st == 0
        plan_equal(plan, oplan)
    # the fixed-order composition on the same buffers is unaffected
    st3, plan3 = p.tg_compose_pipeline(surv, cost, dmax)
    ost3, oplan3, _ = o.compose(o.prune())
    assert st3 == ost3
    if st3 == 0:
        plan_equal(plan3, oplan3)


@pytest.mark.parametrize("name", ["tiny", "dense8b", "dense70b"])
def test_all_orders_named_against_stored(name):
    g = load_golden(name)["all_orders"]
    say("case", name)
    p = T.Problem(load_instance(name))
    surv, cost, dmax = _gpu(p)
    st, plan = p.tg_compose_pipeline_all_orders(surv, cost, dmax)
    assert st == g["status"] == 0
    g["plan"]["status"] = 0
    plan_equal(plan, g["plan"])
    assert plan["T"] == min(row[2] for row in g["per_b"])


def test_all_orders_empty_list_has_no_plan():
    p = T.Problem(load_instance("tiny"))
    _, cost, dmax = _gpu(p)
    st, plan = p.tg_compose_pipeline_all_orders(torch.empty(0, dtype=torch.int64, device="cuda"), cost, dmax)
    assert st == T.TG_ENOPLAN and plan["S"] == 0


def test_all_orders_rejects_more_than_16_islands():
    p = T.Problem(load_instance("moe"))  # 32 islands
    assert T.load_library().tg_compose_all_orders_workspace_bytes(p.h, 0) == 0
    cost = torch.empty(1, dtype=torch.float64, device="cuda")
    dmax = torch.empty(1, dtype=torch.uint8, device="cuda")
    ws = torch.empty(256, dtype=torch.uint8, device="cuda")
    # the library refuses before it reads any buffer (called directly: the
    # binding already refuses score arrays shorter than N)
    vp = ctypes.c_void_p
    plan = T.TgPlan()
    st = T.load_library().tg_compose_pipeline_all_orders(p.h, None, 0, vp(cost.data_ptr()), vp(dmax.data_ptr()),
                                                         ctypes.byref(plan), vp(ws.data_ptr()), ws.numel(), None)
    assert st == T.TG_EINVAL and "16 islands" in T.last_error()
    with pytest.raises(ValueError, match="at least"):
        p.tg_compose_pipeline_all_orders(torch.empty(0, dtype=torch.int64, device="cuda"), cost, dmax,
                                         workspace=ws)
