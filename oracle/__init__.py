"""CPU oracle for the NAMOH routed mixture-of-head attention layer.

TEST INFRASTRUCTURE ONLY.  The test-suite, the smoke check and the
benchmark's CPU-baseline leg are the only code allowed to import anything
from this package.  The GPU library (``paper_2609_38832_amd``) never imports,
calls or links it, and this package imports nothing from the library: the
two share no code.  Only the seeded input generators
(``paper_2609_38832_amd.workloads``, which hold no layer arithmetic) feed
both sides, and they are called by the tests, not from here.

Everything is plain numpy in float64; bf16 inputs are upcast exactly.
See ``namoh_oracle`` for the functions and the paper passages they follow.
"""
from .namoh_oracle import *  # noqa: F401,F403
