"""The compositions read nothing of their workspace that the same call did not
write first.  A workspace is dirtied by a call on a thinned candidate list
(every third survivor dropped: different groups, tables and continuation
rows), then reused for the full surviving set; the plan must equal, bit for
bit, the plan computed on a fresh workspace.  And calls on one handle from
several threads and streams (which share the handle's pinned read-back
words: one call at a time uses them, the others read back another way)
give the single-threaded plan, also with prunes running beside them."""
import threading

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from tests.edge_instances import wide_instance  # noqa: E402
from tests.test_gpu_parity import bits  # noqa: E402
from workloads import load_instance, random_tiny  # noqa: E402

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2606_16907_amd import tangram as T  # noqa: E402


def same_plan(a, b):
    assert (a["b"], a["m"], a["S"]) == (b["b"], b["m"], b["S"])
    for f in ("P", "F", "T"):
        assert bits(a[f]) == bits(b[f]), f
    assert a["stages"] == b["stages"]


def cases():
    out = [(n, lambda n=n: load_instance(n)) for n in ("tiny", "dense8b", "dense70b", "moe")]
    out += [(f"random{s}", lambda s=s: random_tiny(s)) for s in (3, 11)]
    return out


CASES = cases()


@pytest.mark.parametrize("which", ["fixed", "relaxed", "all_orders"])
@pytest.mark.parametrize("name,make", CASES, ids=[c[0] for c in CASES])
def test_dirty_workspace_gives_the_same_plan(name, make, which):
    print("case", name, which, flush=True)
    inst = make()
    p = T.Problem(inst)
    if which == "all_orders" and p.K > 16:
        pytest.skip("all-orders composition takes at most 16 islands")
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    n = int(surv.numel())
    keep = torch.ones(n, dtype=torch.bool, device=surv.device)
    keep[::3] = False
    thin = surv[keep].contiguous()
    call = {"fixed": (p.tg_compose_pipeline, p.compose_workspace),
            "relaxed": (p.tg_compose_pipeline_relaxed, p.compose_relaxed_workspace),
            "all_orders": (p.tg_compose_pipeline_all_orders, p.compose_all_orders_workspace)}[which]
    compose, workspace = call
    fresh_st, fresh = compose(surv, cost, dmax, workspace=workspace(n))
    ws = workspace(n)
    try:  # only dirties the workspace: a thinned list need not give a plan
        compose(thin, cost, dmax, workspace=ws)
    except T.TangramError:
        pass
    st, plan = compose(surv, cost, dmax, workspace=ws)
    torch.cuda.synchronize()
    assert st == fresh_st
    if st == T.TG_OK:
        same_plan(plan, fresh)
    # and once more after a full-list call on the same workspace
    st2, plan2 = compose(surv, cost, dmax, workspace=ws)
    assert st2 == fresh_st
    if st2 == T.TG_OK:
        same_plan(plan2, fresh)
    assert np.isfinite(fresh["T"]) or fresh_st != T.TG_OK


def test_threads_on_one_handle_give_the_same_plan():
    # 70 islands x 70 layers: 70 levels, so the composition reads its fill
    # depth limits back part-way through
    inst = wide_instance(21, 70, 70, "few")
    print("case", inst["name"], flush=True)
    p = T.Problem(inst)
    cost, dmax = p.tg_score_pairs()
    surv = p.tg_prune(cost, dmax)
    n = int(surv.numel())
    ref_st, ref = p.tg_compose_pipeline(surv, cost, dmax)
    torch.cuda.synchronize()
    out, errors = [[], [], []], []

    def worker(k):
        try:
            ws = p.compose_workspace(n)
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.default_stream())
            with torch.cuda.stream(s):
                for _ in range(5):
                    out[k].append(p.tg_compose_pipeline(surv, cost, dmax, workspace=ws))
            s.synchronize()
        except Exception as e:  # reported below, in the test's own thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(k,)) for k in range(3)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for runs in out:
        assert len(runs) == 5
        for st, plan in runs:
            assert st == ref_st
            if st == T.TG_OK:
                same_plan(plan, ref)


def test_prunes_and_compositions_from_threads_share_the_read_back_words():
    """Prunes (survivor count) and compositions (depth limits and plan) on one
    handle from several threads and streams at once: whichever call finds the
    handle's pinned words held reads back another way, and every call returns
    the single-threaded result."""
    inst = wide_instance(21, 70, 70, "few")
    print("case", inst["name"], flush=True)
    p = T.Problem(inst)
    cost, dmax = p.tg_score_pairs()
    ref_surv = p.tg_prune(cost, dmax)
    n = int(ref_surv.numel())
    ref_st, ref = p.tg_compose_pipeline(ref_surv, cost, dmax)
    ref_host = ref_surv.cpu().numpy()
    torch.cuda.synchronize()
    errors, counts = [], []

    def pruner():
        try:
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.default_stream())
            with torch.cuda.stream(s):
                ws = p.prune_workspace()
                buf = torch.empty(n + 64, dtype=torch.int64, device="cuda")
                for _ in range(8):
                    sv = p.tg_prune(cost, dmax, survivors=buf, workspace=ws)
                    counts.append(int(sv.numel()))
                    assert np.array_equal(sv.cpu().numpy(), ref_host)
            s.synchronize()
        except Exception as e:  # reported below, in the test's own thread
            errors.append(e)

    def composer():
        try:
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.default_stream())
            with torch.cuda.stream(s):
                ws = p.compose_workspace(n)
                for _ in range(5):
                    st, plan = p.tg_compose_pipeline(ref_surv, cost, dmax, workspace=ws)
                    assert st == ref_st
                    if st == T.TG_OK:
                        same_plan(plan, ref)
            s.synchronize()
        except Exception as e:
            errors.append(e)

    threads = [threading.Thread(target=f) for f in (pruner, composer, pruner, composer)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    assert counts == [n] * 16
