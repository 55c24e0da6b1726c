"""Co-activation token routing for MoE expert parallelism on MI355X (gfx950).

The routing path of Cobalt ("Leveraging Expert Co-activation for Efficient
Distributed MoE Training"): co-activation statistics, communication-aware
task assignment (Algorithm 1), dispatch layout and pack, and the
gate-weighted combine, as a C ABI (include/cobalt.h) over HIP kernels.

Submodules: binding (ctypes over libcobalt.so), pipeline (one step's
buffers and calls), workload (seeded synthetic inputs), build.
"""
