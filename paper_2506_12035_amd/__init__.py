"""MARche cache-aware decode step on MI355X (gfx950).

The compute path is the C-ABI library ``libmarche.so`` (hand-written HIP
kernels); ``binding`` marshals arguments to it and ``driver`` composes its
calls into decoding steps.  Importing this package loads nothing: the library
is opened on first use and a missing library is an error, never a fallback.
"""
__all__ = ["workload", "schedule", "binding", "driver"]
