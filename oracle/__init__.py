"""CPU oracle for the KV-Direct hot path: TEST INFRASTRUCTURE ONLY.

A plain, slow, fp64 numpy implementation of what the paper defines (Section 3,
"Method"): RMSNorm, the per-head K/V/Q projections, RoPE, the reconstruction
identity and decode attention.  It exists to check the HIP library against the
paper.  Only the tests, the smoke check and the CPU-baseline leg of the benchmark
may import it; the product path never does, and it shares no code with the HIP
library (the two meet only through the seeded input generators, which hold none
of the method's arithmetic).
"""
from .kvdirect import *  # noqa: F401,F403
