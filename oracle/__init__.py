"""CPU oracle of the MOD-DiT hot path (fp64, plain numpy).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check of
__graft_entry__ and by the CPU-baseline leg of bench.py, never by the product
package.  Parity status: every function is pinned by a CPU test against a
value the paper prints, a closed form, a textbook routine, an invariant or
brute force (tests/test_oracle_*.py).
"""
from .moddit_oracle import *  # noqa: F401,F403
from . import moddit_oracle as core  # noqa: F401
