"""Composition of a superset of the surviving set: every compatible candidate
that fits at some depth.  Such a list holds exact ties in (cost, depth) inside
a group (configs with one data-parallel rank differ only in their ZeRO stage,
which then changes neither cost nor memory), so the candidate index decides
between them, and groups longer than a register staircase.  Each composition
must return the plan of the surviving set, and the oracle's plan for the same
superset."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from oracle.oracle import Oracle  # noqa: E402
from tests.test_gpu_parity import plan_equal  # noqa: E402
from tests.test_gpu_workspace import same_plan  # noqa: E402
from workloads import extended, load_instance, random_tiny  # noqa: E402

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2606_16907_amd import tangram as T  # noqa: E402

CASES = [("tiny", lambda: load_instance("tiny")),
         ("random3", lambda: random_tiny(3)),
         ("random11", lambda: random_tiny(11)),
         ("random5_ext", lambda: extended(random_tiny(5), cp=(1, 2), recompute=(0, 1), offload=(0, 1)))]


def superset(p, inst, dmax):
    """Ascending indices of the compatible candidates with d_max >= 1, and
    whether two of them tie in (slice, island, b, cost, d_max)."""
    pairs = p.tg_enumerate_pairs().cpu().numpy().astype(np.int64)
    b = pairs[:, 5] * pairs[:, 10]
    ok = (inst["space"]["global_batch"] % b == 0) & (dmax.cpu().numpy() >= 1)
    idx = np.nonzero(ok)[0].astype(np.int64)
    return idx, pairs[idx], b[idx]


@pytest.mark.parametrize("name,make", CASES, ids=[c[0] for c in CASES])
def test_superset_composes_to_the_surviving_plan(name, make):
    print("case", name, flush=True)
    inst = make()
    p = T.Problem(inst)
    o = Oracle(inst)
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    idx, pairs, b = superset(p, inst, dmax)
    assert len(idx) > surv.numel()
    # exact ties present: the same group, cost and depth for two candidates
    key = np.stack([pairs[:, 0], pairs[:, 1], pairs[:, 2], b,
                    cost.cpu().numpy()[idx].view(np.int64), dmax.cpu().numpy()[idx].astype(np.int64)], axis=1)
    assert len(np.unique(key, axis=0)) < len(key)
    sup = torch.from_numpy(idx).cuda()
    calls = [("fixed", p.tg_compose_pipeline, o.compose),
             ("relaxed", p.tg_compose_pipeline_relaxed, o.compose_relaxed)]
    if p.K <= 16:
        calls.append(("all_orders", p.tg_compose_pipeline_all_orders, o.compose_all_orders))
    for which, gpu, orc in calls:
        print("  ", which, len(idx), "candidates", flush=True)
        st_s, plan_s = gpu(surv, cost, dmax)
        st_x, plan_x = gpu(sup, cost, dmax)
        torch.cuda.synchronize()
        assert st_x == st_s
        ost, oplan = orc(idx)[:2]
        assert st_x == ost
        if st_x == T.TG_OK:
            same_plan(plan_x, plan_s)
            plan_equal(plan_x, oplan)
