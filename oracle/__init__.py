"""fp64 CPU oracle and comparison rule.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU baseline, never by the product path.  Shares no code with
the HIP library.
"""
from . import compare, kbest_oracle  # noqa: F401
