"""GPU parity at the edges of the supported sizes (tests/edge_instances.py):
every candidate's score bit for bit, the surviving set, and the plans of both
compositions, against the live oracle."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from oracle.oracle import Oracle  # noqa: E402
from tests.edge_instances import EDGE_CASES, wide_instance  # noqa: E402
from tests.test_gpu_parity import bits, plan_equal  # noqa: E402

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2606_16907_amd import tangram as T  # noqa: E402


@pytest.mark.parametrize("seed,K,L,links", EDGE_CASES,
                         ids=[f"K{k}_L{l}_{e}" for _, k, l, e in EDGE_CASES])
def test_edge_parity(seed, K, L, links):
    inst = wide_instance(seed, K, L, links, tight=(seed % 2 == 0))
    print("case", inst["name"], links, flush=True)
    sys.stdout.flush()
    o = Oracle(inst)
    p = T.Problem(inst)
    assert (p.N, p.NS, p.n_configs, p.n_b) == (o.N, o.NS, o.n_configs, o.n_b)
    cost, dmax = p.tg_score_pairs()
    oc, od = o.score()
    torch.cuda.synchronize()
    assert np.array_equal(bits(cost.cpu().numpy()), bits(oc))
    assert np.array_equal(dmax.cpu().numpy(), od)
    surv = p.tg_prune(cost, dmax)
    osurv = o.prune()
    assert np.array_equal(surv.cpu().numpy(), osurv)
    st, plan = p.tg_compose_pipeline(surv, cost, dmax)
    ost, oplan, _ = o.compose(osurv)
    assert st == ost
    if st == 0:
        plan_equal(plan, oplan)
    st, plan = p.tg_compose_pipeline_relaxed(surv, cost, dmax)
    ost, oplan, _ = o.compose_relaxed(osurv)
    assert st == ost
    if st == 0:
        plan_equal(plan, oplan)
