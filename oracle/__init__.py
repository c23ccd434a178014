"""CPU oracle for the FP8 speculative-verify path.

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import, call, link or execute anything in
this package.  The product path (paper_2606_18502_amd) never touches it, and
this package never imports the product package: the two share no code, no
tables and no constants.  The only common module is `workloads`, which draws
the seeded synthetic inputs and holds none of the method's arithmetic.

Everything here is written to be checked by eye against its definition:
numpy in fp64 (exact where the definition allows), plain Python loops for the
sequential parts, Fractions for the exact-enumeration proofs.

Parity pins: every function in this package is pinned by the CPU tests in
tests/test_oracle_*.py against something other than itself (the E4M3 format
definition and torch's independent float8_e4m3fn cast, closed-form error
bounds, integer-exact GEMMs, one-hot selections, exact Fraction enumeration of
the speculative-sampling law, the closed-form expected acceptance length).
"""

from . import e4m3, quantize, gemm, accept, enumerate, kvcache  # noqa: F401
