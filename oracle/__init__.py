"""fp64 CPU oracle for MARche's cache-aware decode step -- TEST INFRASTRUCTURE.

Only the test suite, the smoke check and the CPU-baseline leg of the benchmark
may import this package.  The product path (the HIP library and its Python
binding) never calls it and shares no code with it.

Everything here is plain numpy in float64, per image, written to be read
against the paper:

* ``block``    -- the pre-LN bidirectional block; cache-aware attention
                  (Algorithm 1, Section 4.1) in the single-pass form and in
                  Appendix A's two-segment form; the per-key attention mass of
                  the generating rows (Section 4.2).
* ``select``   -- top-k refresh selection (Section 4.2) and the active-token
                  budget (Section 4.3), plus a brute-force twin.
* ``schedule`` -- the mask schedule and the generating / caching token sets
                  (Section 3, Eq. 1-4) and the full-refresh rules (Section 4.3).
* ``step``     -- one MARche decoding step over a stack of blocks.
* ``mar``      -- the rest of a MAR step around the decoder: encoder input and
                  encoder (Eq. 1), decoder input (Eq. 2), the condition and
                  the DDPM sampler of Eq. 3.

Parity status per function is listed in each module's header.
"""
from . import block, mar, schedule, select, step  # noqa: F401
