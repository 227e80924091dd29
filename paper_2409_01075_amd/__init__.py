"""vx: runtime-shaped dense GEMM for MI355X (gfx950).

The compute path is the HIP library ``libvx.so`` (C ABI in include/vx.h);
``paper_2409_01075_amd.vx`` binds it.  ``paper_2409_01075_amd.inputs`` holds
the seeded workload generators.
"""
__all__ = ["vx", "inputs"]
