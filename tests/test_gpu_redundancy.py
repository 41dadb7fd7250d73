"""Parity of the HIP path with redundancy pruning (tg_score_classes,
tg_prune_classes, tg_compose_pipeline_classes, through the C ABI) with the
CPU oracle: the class count, each class's scores (those of its first slice,
scored by the oracle), the surviving set bit for bit (the oracle's, with and
without redundancy pruning), and the composed plan; on random instances with
repeated layers, imbalance pruning and the extended space, and on the 70B,
MoE and 128-island instances against the oracle's stored survivor digests
and plans."""
import copy
import hashlib
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from oracle.oracle import Oracle  # noqa: E402
from workloads import extended, load_instance  # noqa: E402
from tests.inst_util import tiny_tight  # noqa: E402
from tests.golden.make_golden import load as load_golden  # noqa: E402
from tests.test_gpu_parity import bits, plan_equal  # noqa: E402
from tests.test_oracle_redundancy import _random  # noqa: E402

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2606_16907_amd import tangram as T  # noqa: E402


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _eps(inst, eps):
    out = copy.deepcopy(inst)
    out["space"]["imbalance_eps"] = eps
    return out


CASES = ([(f"rand{s}", lambda s=s: _random(s)) for s in range(16)]
         + [(f"rand_imb{s}", lambda s=s: _eps(_random(s), 0.5)) for s in (0, 4, 8)]
         + [("tiny", lambda: load_instance("tiny")), ("tiny_tight", tiny_tight),
            ("dense8b", lambda: load_instance("dense8b")),
            ("dense8b_ext", lambda: extended(load_instance("dense8b")))])


@pytest.mark.parametrize("name,make", CASES, ids=[n for n, _ in CASES])
def test_redundancy_parity(name, make):
    inst = make()
    say("case", name)
    o = Oracle(inst)
    cls, nc = o.slice_classes()
    p = T.Problem(inst)
    assert p.NC == nc
    cost_c, dmax_c = p.tg_score_classes()
    # class candidate (g, c) scores the class's first slice
    first = np.array([list(cls).index(c) for c in range(nc)], dtype=np.int64)
    idx = (np.arange(o.n_configs, dtype=np.int64)[:, None] * o.NS + first[None, :]).reshape(-1)
    oc, od = o.score_list(idx)
    assert np.array_equal(bits(cost_c.cpu().numpy()), bits(oc))
    assert np.array_equal(dmax_c.cpu().numpy(), od)
    surv = p.tg_prune_classes(cost_c, dmax_c)
    want = o.prune()
    assert np.array_equal(surv.cpu().numpy(), want)
    assert np.array_equal(want, o.prune_classes())
    st, plan = p.tg_compose_pipeline_classes(surv, cost_c, dmax_c)
    ost, oplan, _ = o.compose(want)
    if ost != 0:
        assert st == T.TG_ENOPLAN
    else:
        assert st == 0
        plan_equal(plan, oplan)


@pytest.mark.parametrize("name", ["dense70b", "moe", "large"])
def test_redundancy_named_against_stored(name):
    g = load_golden(name)
    say("case", name)
    p = T.Problem(load_instance(name))
    assert p.NC == p.L  # uniform decoder layers: one class per slice length
    cost_c, dmax_c = p.tg_score_classes()
    surv = p.tg_prune_classes(cost_c, dmax_c)
    s = surv.cpu().numpy()
    assert len(s) == g["survivors"]["count"]
    assert hashlib.sha256(np.ascontiguousarray(s, dtype="<i8").tobytes()).hexdigest() == g["survivors"]["sha256"]
    st, plan = p.tg_compose_pipeline_classes(surv, cost_c, dmax_c)
    assert st == g["status"] == 0
    g["plan"]["status"] = 0
    plan_equal(plan, g["plan"])
