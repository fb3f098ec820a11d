"""Fork-aware decode attention for gfx950 (MI355X).

The compute lives in ``libforkattn.so`` (HIP kernels behind a C ABI declared in
``include/forkattn.h``); ``forkattn`` is its thin ctypes binding and
``workloads`` draws the seeded synthetic inputs.  Importing the package loads
nothing: ``from paper_2608_13667_amd import forkattn`` loads the library and
fails loudly when it has not been built.
"""
__all__ = ["forkattn", "workloads"]
