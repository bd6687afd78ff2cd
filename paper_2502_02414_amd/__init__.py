"""MI355X (gfx950) Physics-Attention hot path of Transolver++ (arXiv 2502.02414).

The layer's arithmetic lives in hand-written HIP kernels behind the C-ABI
library ``libpa.so`` (declared in ``include/pa.h``).  ``binding`` wraps those
entry points with the same names for torch device tensors; ``inputs`` draws
the seeded synthetic workloads.  Importing the package loads nothing.
"""
__all__ = ["binding", "inputs"]
