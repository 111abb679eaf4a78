"""DeltaLog decode state update for MI355X (gfx950).

The hot path lives in ``libdeltalog.so`` (hand-written HIP kernels behind a C ABI,
declared in ``include/deltalog.h``).  ``paper_2608_15533_amd.deltalog`` is the thin
ctypes binding with the same entry-point names; importing it loads the library and
fails loudly if it has not been built (``python -m paper_2608_15533_amd.build``).

Submodules are imported on demand so that the pure-host helpers (``workloads``,
``traffic``) can be used without the compiled library.
"""

__all__ = ["deltalog", "workloads", "traffic", "build"]
