"""CPU oracle for CRISP sparse prefill attention -- TEST INFRASTRUCTURE ONLY.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this package.  The product path (the HIP library and its binding) never imports
it and fails loudly when its extension is missing.

Parity status of each function is recorded in tests/test_oracle_pins.py: every
stage is pinned by a closed form, an invariant, a library routine or brute force.
"""
from .crisp_oracle import *  # noqa: F401,F403
from .crisp_oracle import Params, HeadResult, ROUTE_VS, ROUTE_PE  # noqa: F401
