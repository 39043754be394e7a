"""Plain fp64 CPU oracle for the routed mixture-of-experts layer.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call,
link or execute this package: only the test suite, the smoke check in
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` use it.
It shares no code with the HIP library: no kernels, headers, helpers,
tables or pre/post-processing. Both sides only consume the seeded inputs
written by the separate ``synth`` package.

Modules
-------
mx   -- bit-level definitions of the FP4 (e2m1) weight codes, the E8M0 block
        scales and the MX activation formats, plus the per-32 activation
        quantiser.
moe  -- the layer: top-k routing, stable token->expert permutation,
        activation quantisation, gate/up -> SwiGLU -> down expert FFN, and the
        weighted combine.

Pins (values fixed by the paper or by mathematics, not by this code) live in
``tests/test_oracle_*.py``; every function here is pinned by at least one of
them (see the per-function docstrings).
"""
from . import mx, moe  # noqa: F401
