"""MI355X-native INT8 encoder-decoder inference engine (MobileNMT, arXiv 2306.04235).

The engine is the C-ABI shared library ``libmnmt.so`` built from ``csrc/``
(HIP kernels for gfx950 plus the host-side loader, planner and drivers);
``mnmt`` is its thin Python binding.  Importing this package does not load
the library; ``mnmt.lib()`` does, and raises if it has not been built.
"""
__all__ = ["mnmt", "workload"]
