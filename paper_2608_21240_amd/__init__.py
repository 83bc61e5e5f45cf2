"""SPICE MoE-layer hot path for AMD Instinct MI355X (gfx950).

    spice     -- ctypes binding of libspice_moe.so (C ABI in include/spice_moe.h)
    layer     -- driver of one layer call (device memory, streams, host staging)
    synth     -- seeded synthetic inputs
    workloads -- layer shapes and workload settings
    build     -- compiles libspice_moe.so with hipcc for gfx950

Submodules are imported on demand so that importing the package touches
neither torch nor the GPU.
"""
