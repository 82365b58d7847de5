"""Page-centric sparse decode attention for MI355X (gfx950), after Vortex (arXiv 2606.06453).

The hot path lives in ``libvx.so`` (hand-written HIP kernels behind a C ABI, declared in
``include/vx.h``); :mod:`paper_2606_06453_amd.vx` is the thin ctypes binding.  The binding is
imported lazily so that :mod:`paper_2606_06453_amd.workloads` can be used without a GPU.
"""
__all__ = ["vx", "workloads"]
