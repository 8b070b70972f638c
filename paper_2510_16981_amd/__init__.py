"""MI355X (gfx950) implementation of the MuonBP optimizer step.

The step runs in ``libmuonbp.so`` (hand-written HIP kernels behind a C ABI,
declared in ``include/muonbp.h``).  ``paper_2510_16981_amd.muonbp`` is the
ctypes binding; it is imported lazily so that the input generators in
``paper_2510_16981_amd.workload`` can be used without the library.
"""

__all__ = ["workload"]
