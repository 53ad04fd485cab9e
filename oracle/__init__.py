"""Plain, slow CPU oracle for the delayed-scaling FP8 linear layer with split backward.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only the tests, the smoke check and the CPU-baseline leg
of the benchmark use it.  It shares no code with the HIP library (no kernels,
headers, helpers, tables or constant generators); the only thing the two sides
have in common is the seeded input generator in ``workloads.py``, which holds
none of the method's arithmetic.

What it computes, and where the paper states it:

* ``fp8``       OCP-style E4M3 / E5M2 encode and decode (the paper uses FP8
                without naming encodings; §2.1 cites the FP8-formats paper that
                defines them).  Round to nearest even, saturating.
* ``scaling``   per-tensor amax recording and the delayed scale update from a
                rolling amax history (§2.1; the state S of the §3.2 transition
                equations).
* ``gemm``      quantize, and the three GEMMs of the split layer:
                Y = X W^T (F), dX = dY W (dI), dW = dY^T X (dW) on FP8 codes,
                accumulated in float64 (§3.2 transition equations), plus the
                affine placement of dW into a flat FP32 main-gradient buffer
                (§3.4, §4.3 arena capacity).
* ``contract``  the bookkeeping state machine: TapeKey / TapeRef with slot
                generations (§3.1), effect token (§3.2), weight and cache
                versions (§3.3), arena bindings and exactly-once writes (§3.4),
                Algorithm 1 and the failure rules of §4.5 and Table "faults".
* ``layer``     a stage of FP8 linears that runs F / dI / dW actions through
                the contract and the numerics above, in schedule order.

Functions that have no independent pin say "parity unpinned" in their docstring.
"""
from . import fp8, scaling, gemm, contract, layer  # noqa: F401
