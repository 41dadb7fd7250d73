"""The score kernel's depth rule where its first guess is wrong.  The guess
floor((H - state) * tp/mb * (1 / Act)) can land one below the answer when the
memory limit is met exactly: with 49-byte activation stashes per layer and no
parameters (state 0), islands of 49 * N bytes hold a slice of k layers at
micro-batch mb and tensor degree tp up to exactly depth N * tp / (mb * k),
while 49 * fl(1/49) < 1 in binary64.  Every candidate's cost and depth must
equal the oracle's bit for bit, and some live candidates must have had a
wrong guess (so the wave's walk ran, mixed with lanes whose guess was
right)."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

from oracle.oracle import Oracle  # noqa: E402
from tests.inst_util import instance  # noqa: E402
from tests.test_gpu_parity import bits  # noqa: E402

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

from paper_2606_16907_amd import tangram as T  # noqa: E402


def boundary_instance(L, K, N, tp, mb):
    layer = {"fwd_flops": 10**12, "act_stash_bytes": 49, "tp_comm_bytes": 10**6, "out_act_bytes": 10**6}
    return instance(L=L, K=K, layer=layer, n_gpus=8, hbm=float(49 * N), B=4096, tp=tp, mb=mb,
                    zero=(0, 1, 2, 3), mem_frac=1.0)


def wrong_guesses(p, inst, dmax):
    """Live candidates whose first guess differs from their depth (the guess
    taken in the kernel's operation order: (H - state) * (q / mb) * (1 / Act),
    state 0 here)."""
    pairs = p.tg_enumerate_pairs().cpu().numpy().astype(np.int64)
    i, j, tp, cp, mb = pairs[:, 0], pairs[:, 1], pairs[:, 3], pairs[:, 4], pairs[:, 10]
    H = np.float64(inst["islands"]["hbm_bytes"][0]) * np.float64(inst["space"]["mem_frac"])
    act = (49 * (j - i)).astype(np.float64)
    inv_rho = (tp * cp).astype(np.float64) / mb.astype(np.float64)
    q = (H - 0.0) * (inv_rho * (1.0 / act))
    b = pairs[:, 5] * mb
    m = np.float64(inst["space"]["global_batch"]) / b.astype(np.float64)
    K = p.K
    g = np.where(q >= m, K, np.floor(np.clip(q, 0, K))).astype(np.int64)
    return int(np.count_nonzero(g != dmax.cpu().numpy().astype(np.int64)))


@pytest.mark.parametrize("L,K,N,tp,mb", [(24, 8, 24, (1, 2), (1, 2, 4)),
                                          (30, 12, 60, (1, 2, 4), (1, 2, 3)),
                                          (70, 16, 840, (1, 2, 4, 8), (1, 2, 4, 8))])
def test_depth_rule_where_the_guess_is_wrong(L, K, N, tp, mb):
    inst = boundary_instance(L, K, N, tp, mb)
    print("case", L, K, N, tp, mb, flush=True)
    p = T.Problem(inst)
    o = Oracle(inst)
    cost, dmax = p.tg_score_pairs()
    oc, od = o.score()
    torch.cuda.synchronize()
    assert np.array_equal(bits(cost.cpu().numpy()), bits(oc))
    assert np.array_equal(dmax.cpu().numpy(), od)
    assert wrong_guesses(p, inst, dmax) > 0
    # and the path after scoring on these depths
    surv = p.tg_prune(cost, dmax)
    assert np.array_equal(surv.cpu().numpy(), o.prune())
