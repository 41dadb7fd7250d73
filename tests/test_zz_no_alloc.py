"""tg_prune_no_alloc (the surviving set on the library's static scratch,
for callers that cannot allocate) against tg_prune with a workspace, through
the C ABI: the same ascending survivor list, bit for bit, on calls in a row
whose problems shrink (the 128-island instance, the 80-layer one, the 8-layer
one), so the second and third calls run on scratch the larger call left
behind; and the refusal of a problem whose workspace exceeds the scratch."""
import ctypes

import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu


def _require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


def test_no_alloc_prune_equals_prune_on_shrinking_calls():
    _require_gpu()
    from paper_2606_16907_amd import tangram as T
    from workloads import load_instance
    torch.cuda.set_device(0)
    lib = T.load_library()
    for name in ("large", "dense70b", "tiny"):
        print(f"no-alloc prune: {name}", flush=True)
        p = T.Problem(load_instance(name))
        assert lib.tg_prune_workspace_bytes(p.h) <= 64 << 20
        cost, dmax = p.tg_score_pairs()
        ref = p.tg_prune(cost, dmax)
        n_ref = int(ref.numel())
        buf = torch.full((n_ref + 64,), -7, dtype=torch.int64, device="cuda")
        got = p.tg_prune_no_alloc(cost, dmax, buf)
        torch.cuda.synchronize()
        assert int(got.numel()) == n_ref
        assert torch.equal(got, ref), name
        assert bool((buf[n_ref:] == -7).all()), "wrote past the survivor count"
        # capacity too small: the count, TG_ECAPACITY, nothing past capacity
        small = torch.full((max(n_ref // 2, 1),), -7, dtype=torch.int64, device="cuda")
        with pytest.raises(T.TangramError) as e:
            p.tg_prune_no_alloc(cost, dmax, small)
        assert e.value.status == T.TG_ECAPACITY and e.value.required == n_ref
        torch.cuda.synchronize()
        assert torch.equal(small, ref[: small.numel()])
        del p, cost, dmax, ref, buf, got, small
        torch.cuda.empty_cache()


def test_no_alloc_prune_refuses_a_workspace_beyond_the_scratch():
    _require_gpu()
    from paper_2606_16907_amd import tangram as T
    from workloads import extended, load_instance
    torch.cuda.set_device(0)
    lib = T.load_library()
    p = T.Problem(extended(load_instance("large")))
    need = lib.tg_prune_workspace_bytes(p.h)
    assert need > 64 << 20
    n = ctypes.c_int64(-1)
    # refused on the size alone, before any pointer is used or work is queued
    st = lib.tg_prune_no_alloc(p.h, ctypes.c_void_p(8), ctypes.c_void_p(8), ctypes.c_void_p(8), 1,
                               ctypes.byref(n), None)
    assert st == T.TG_ENOMEM
    assert "static scratch" in T.last_error()
