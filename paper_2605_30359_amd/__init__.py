"""kf: fused contraction + epilogue kernels for AMD MI355X (gfx950).

The compute path is the C-ABI library ``libkf.so`` (hand-written HIP kernels);
``paper_2605_30359_amd.kf`` is its thin ctypes binding.  ``inputs`` holds the
seeded workload generators.  Submodules are imported on demand so that
``inputs`` can be used without loading the GPU library.
"""
__all__ = ["inputs", "kf"]
