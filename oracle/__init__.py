"""CPU oracle for one routed MoE layer.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
link this package: only the tests, the smoke check and the benchmark's CPU
baseline leg use it.  It shares no code, header, table or helper with the HIP
library; both sides receive their inputs from the seeded generators alone.

Every public function is pinned by a CPU test against something other than
itself (brute force, closed forms, invariants, printed values); see
``moe_oracle`` for the list.  No function is "parity unpinned".
"""
from .moe_oracle import *  # noqa: F401,F403
