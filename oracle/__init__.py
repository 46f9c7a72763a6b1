"""Oracle for the partial-straggler gradient-coding hot path.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, fp64 CPU
implementation of what the hot path computes, written from the paper
("Leveraging partial stragglers within gradient coding", Ramamoorthy, Meng,
Girimaji).  Only the test suite, the smoke check and the benchmark's CPU
baseline leg may import it.  It shares no code with the HIP library and never
imports it; both consume the same stored inputs from ``workloads``.

Modules:
    assignment  cyclic assignment, ordering matrix O and its tables (Sec. 1, Sec. 3)
    gradients   per-chunk gradients g_{D_i} (Sec. 1)
    protocol    processed sets, coverage, decodability, Algorithm 1, encode,
                PS combine (Sec. 2, Sec. 2.1, Sec. 2.2)
    ordering    Algorithm 2, chunk ordering of regular assignments (Sec. 3)
    simulation  worker progress and exact-GC completion times (Sec. 4)
"""
from . import assignment, gradients, ordering, protocol, simulation  # noqa: F401
