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
