"""ART (Attention Run-time Termination) decode attention for MI355X (gfx950).

The computation lives in libart.so (HIP kernels behind the C ABI of
include/art.h); ``paper_2606_00024_amd.api`` is the PyTorch-facing binding,
``paper_2606_00024_amd.workloads`` the seeded synthetic input generator and
``paper_2606_00024_amd.build`` the in-tree build.  Importing the package loads
nothing: the library is loaded on first use and its absence is an error.
"""

__all__ = ["api", "workloads", "build"]
