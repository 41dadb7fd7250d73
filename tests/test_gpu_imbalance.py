"""Parity of the HIP path with imbalance pruning on (tg_space.imbalance_eps,
through the C ABI) with the CPU oracle: the surviving set bit for bit, and
the plans of the fixed-order, relaxed and all-orders compositions, on random
instances (where pruning leaves holes before the first balanced cut, so the
compositions' cut scans must start there), on the small named instances
live, and on the 70B, MoE and 128-island instances against the oracle's
stored results; a list holding an unbalanced pair is rejected."""
import copy
import hashlib
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from oracle.oracle import Oracle  # noqa: E402
from workloads import load_instance, random_tiny  # noqa: E402
from tests.inst_util import instance  # noqa: E402
from tests.golden.make_golden import load as load_golden  # noqa: E402
from tests.test_gpu_parity import plan_equal  # noqa: E402

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2606_16907_amd import tangram as T  # noqa: E402


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def with_eps(inst, eps):
    out = copy.deepcopy(inst)
    out["space"]["imbalance_eps"] = float(eps)
    return out


CASES = ([(f"rand{s}", lambda s=s: with_eps(random_tiny(s, tight=(s % 2 == 1)), (0.25, 0.5, 1.0)[s % 3]))
          for s in range(24)]
         + [(f"randL{s}", lambda s=s: with_eps(random_tiny(1000 + s, L_range=(9, 14), K_range=(3, 6)), 1.0))
            for s in range(6)]
         + [("tiny", lambda: with_eps(load_instance("tiny"), 0.5)),
            ("dense8b", lambda: with_eps(load_instance("dense8b"), 0.5))])


def _check_plan(st, plan, ost, oplan):
    if ost != 0:
        assert st == T.TG_ENOPLAN and plan["S"] == 0
    else:
        assert st == 0
        plan_equal(plan, oplan)


@pytest.mark.parametrize("name,make", CASES, ids=[n for n, _ in CASES])
def test_imbalance_parity(name, make):
    inst = make()
    say("case", name)
    o = Oracle(inst)
    os_ = o.prune()
    p = T.Problem(inst)
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    assert np.array_equal(surv.cpu().numpy(), os_)
    st, plan = p.tg_compose_pipeline(surv, cost, dmax)
    _check_plan(st, plan, *o.compose(os_)[:2])
    st, plan = p.tg_compose_pipeline_relaxed(surv, cost, dmax)
    _check_plan(st, plan, *o.compose_relaxed(os_)[:2])
    if o.K <= 16:
        st, plan = p.tg_compose_pipeline_all_orders(surv, cost, dmax)
        _check_plan(st, plan, *o.compose_all_orders(os_)[:2])


@pytest.mark.parametrize("name", ["dense70b", "moe", "large"])
def test_imbalance_named_against_stored(name):
    g = load_golden(name + "_imbalance")
    say("case", name, "eps", g["imbalance_eps"])
    p = T.Problem(with_eps(load_instance(name), g["imbalance_eps"]))
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    s = surv.cpu().numpy()
    assert len(s) == g["survivors"]["count"]
    assert s[:16].tolist() == g["survivors"]["head"] and s[-16:].tolist() == g["survivors"]["tail"]
    assert hashlib.sha256(np.ascontiguousarray(s, dtype="<i8").tobytes()).hexdigest() == g["survivors"]["sha256"]
    st, plan = p.tg_compose_pipeline(surv, cost, dmax)
    assert st == g["status"] == 0
    g["plan"]["status"] = 0
    plan_equal(plan, g["plan"])


def test_unbalanced_pair_rejected():
    inst = with_eps(instance(K=2, L=8, layer={"fwd_flops": 2 ** 40}, n_gpus=[3, 1], B=4, tp=(1,), mb=(1,),
                             zero=(0,)), 0.5)
    p = T.Problem(inst)
    cost, dmax = p.tg_score_pairs()
    bad = torch.tensor([0], dtype=torch.int64, device="cuda")  # slice [0, 1) on island 0: 1/8 vs 3/4
    for call in (p.tg_compose_pipeline, p.tg_compose_pipeline_all_orders):
        with pytest.raises(T.TangramError) as e:
            call(bad, cost, dmax)
        assert e.value.status == T.TG_EINVAL
