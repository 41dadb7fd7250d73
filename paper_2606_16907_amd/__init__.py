"""MI355X (gfx950) plan search of Tangram's heterogeneous planner.

The hot path (scoring of every model-slice/island/config candidate, pruning,
pipeline composition) runs in the HIP library libtangram_hip.so behind the C
ABI of include/tangram.h; the submodule `tangram` is its ctypes binding and
`build` compiles the library.
"""
