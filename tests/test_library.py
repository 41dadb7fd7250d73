"""The built HIP library loads on the CPU host and exports every symbol the
C header declares (no compute calls: those need the GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tangram.h")
LIB = os.path.join(ROOT, "paper_2606_16907_amd", "libtangram_hip.so")


def declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tg_[a-z_]+)\s*\(", text)))


def test_header_declares_the_four_entry_points():
    names = declared()
    for n in ("tg_enumerate_pairs", "tg_score_pairs", "tg_prune", "tg_compose_pipeline"):
        assert n in names


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(LIB)
    missing = [n for n in declared() if not hasattr(lib, n)]
    assert not missing, missing


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_binding_declares_every_export():
    from paper_2606_16907_amd import tangram as T
    assert sorted(T.EXPORTS) == declared()
    T.load_library()


def test_binding_struct_layouts_match_header_sizes():
    from paper_2606_16907_amd import tangram as T
    assert ctypes.sizeof(T.TgLayer) == 64
    assert ctypes.sizeof(T.TgIsland) == 40
    assert ctypes.sizeof(T.TgSpace) == 200
    assert ctypes.sizeof(T.TgPair) == 48
    assert ctypes.sizeof(T.TgStage) == 80
    assert ctypes.sizeof(T.TgPlan) == 16 + 24 + 255 * 80


def test_struct_sizes_agree_with_the_c_compiler(tmp_path):
    import subprocess
    from paper_2606_16907_amd import tangram as T
    src = tmp_path / "sizes.c"
    src.write_text('#include <stdio.h>\n#include "tangram.h"\nint main(void){printf("%zu %zu %zu %zu %zu '
                   '%zu %zu\\n", sizeof(tg_layer), sizeof(tg_island), sizeof(tg_space), '
                   'sizeof(tg_pair), sizeof(tg_stage), sizeof(tg_plan), sizeof(tg_info));return 0;}\n')
    exe = tmp_path / "sizes"
    subprocess.check_call(["gcc", "-I", os.path.join(ROOT, "include"), "-o", str(exe), str(src)])
    got = [int(x) for x in subprocess.check_output([str(exe)]).split()]
    want = [ctypes.sizeof(c) for c in (T.TgLayer, T.TgIsland, T.TgSpace, T.TgPair, T.TgStage,
                                       T.TgPlan, T.TgInfo)]
    assert got == want


def _space(T, mb, zero_mask=0xF, recompute_mask=0, offload_mask=0):
    sp = T.TgSpace()
    sp.global_batch = 1024
    sp.n_tp, sp.tp[0] = 1, 1
    sp.n_ep, sp.ep[0] = 1, 1
    sp.n_mb = len(mb)
    for a, v in enumerate(mb):
        sp.mb[a] = v
    sp.zero_mask = zero_mask
    sp.recompute_mask, sp.offload_mask = recompute_mask, offload_mask
    sp.eta, sp.mem_frac = 0.5, 0.9
    return sp


def _create(T, lib, n_gpus, sp):
    layers = (T.TgLayer * 2)()
    for y in layers:
        y.fwd_flops, y.dense_params, y.out_act_bytes = 10**9, 10**6, 10**5
    isl = (T.TgIsland * 1)()
    isl[0].n_gpus, isl[0].peak_flops, isl[0].hbm_bytes = n_gpus, 1e15, 1e11
    isl[0].intra_bw, isl[0].host_bw = 1e11, 1e10
    bw = (ctypes.c_double * 1)(0.0)
    out = ctypes.c_void_p(123)
    st = lib.tg_problem_create(layers, 2, isl, 1, bw, ctypes.byref(sp), ctypes.byref(out))
    return st, out.value, lib.tg_last_error().decode()


def test_create_refuses_a_config_space_of_2_23_configs_before_any_device_call():
    """65536 GPUs x 4 ZeRO stages x 2 recompute x 2 offload x 8 micro-batch
    sizes = 2^23 configs, one more than the 23-bit member index holds: the
    counting pass refuses it before the tables (1.6 GB of config rows) or
    any device call.  Validation only, so it runs without a GPU."""
    import time
    from paper_2606_16907_amd import tangram as T
    lib = T.load_library()
    sp = _space(T, [1, 2, 4, 8, 16, 32, 64, 128], recompute_mask=3, offload_mask=3)
    t0 = time.perf_counter()
    st, out, msg = _create(T, lib, 65536, sp)
    assert st == -1 and out is None, (st, msg)
    assert "too large" in msg
    assert time.perf_counter() - t0 < 5.0


def test_create_validation_errors_leave_out_null():
    from paper_2606_16907_amd import tangram as T
    lib = T.load_library()
    sp = _space(T, [1, 2])
    sp.reserved = 1
    st, out, msg = _create(T, lib, 8, sp)
    assert st == -1 and out is None and "reserved" in msg
    sp = _space(T, [2, 1])  # not ascending
    st, out, msg = _create(T, lib, 8, sp)
    assert st == -1 and out is None and "mb set" in msg
    st, out, msg = _create(T, lib, 0, _space(T, [1]))
    assert st == -1 and out is None and "n_gpus" in msg


def test_create_refuses_plans_whose_b_or_m_overflow_int32():
    """A plan reports b and m = B / b as int32: a global batch whose smallest
    compatible b leaves B / b >= 2^31 is refused at create (validation only,
    before any device call)."""
    from paper_2606_16907_amd import tangram as T
    lib = T.load_library()
    sp = _space(T, [1])
    sp.global_batch = 1 << 31  # b = 1 divides it, m = 2^31
    st, out, msg = _create(T, lib, 8, sp)
    assert st == -1 and out is None and "2^31" in msg, (st, msg)


def test_create_takes_islands_of_up_to_2_28_gpus():
    """Islands from tg_build_islands sum their nodes' GPUs (4096 nodes of at
    most 65536): create accepts n_gpus up to 2^28 and refuses more.  At 2^28
    the space itself is refused as too large, which is validation, not the
    GPU count."""
    from paper_2606_16907_amd import tangram as T
    lib = T.load_library()
    st, out, msg = _create(T, lib, (1 << 28) + 1, _space(T, [1]))
    assert st == -1 and out is None and "n_gpus" in msg
    st, out, msg = _create(T, lib, 1 << 28, _space(T, [1]))
    assert st == -1 and out is None and "too large" in msg, msg


class _FakeTensor:
    """Just the attributes the binding's buffer checks read."""

    def __init__(self, dtype, n, cuda=True, contiguous=True, index=0, esize=1):
        import types
        self.dtype, self._n, self.is_cuda, self._c, self._e = dtype, n, cuda, contiguous, esize
        self.device = types.SimpleNamespace(index=index)

    def is_contiguous(self):
        return self._c

    def numel(self):
        return self._n

    def element_size(self):
        return self._e

    def data_ptr(self):
        return 4096


def test_binding_refuses_buffers_the_kernels_would_overrun():
    """The C ABI takes plain pointers, so the binding checks each caller
    buffer (device, dtype, contiguity, length) before any call."""
    import torch
    from paper_2606_16907_amd import tangram as T
    f64 = torch.float64
    ok = T._dbuf(_FakeTensor(f64, 10), f64, 10, "cost", 0)
    assert ok.value == 4096
    bad = [(None, "device buffer"),
           (_FakeTensor(f64, 10, cuda=False), "device buffer"),
           (_FakeTensor(torch.float32, 10), "dtype"),
           (_FakeTensor(f64, 10, contiguous=False), "contiguous"),
           (_FakeTensor(f64, 10, index=1), "cuda:1"),
           (_FakeTensor(f64, 9), "at least 10")]
    for t, msg in bad:
        with pytest.raises(ValueError, match=msg):
            T._dbuf(t, f64, 10, "cost", 0)
    ptr, nbytes = T._dws(_FakeTensor(torch.int64, 5, esize=8), "workspace", 0)
    assert ptr.value == 4096 and nbytes == 40
    for t in (None, _FakeTensor(torch.uint8, 5, contiguous=False), _FakeTensor(torch.uint8, 5, index=2)):
        with pytest.raises(ValueError):
            T._dws(t, "workspace", 0)
