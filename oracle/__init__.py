"""CPU oracle of the PPD verification step (float64 numpy).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the GPU library, with which it shares no
code.  Parity status of each function is listed in its docstring; all are
pinned by CPU tests against brute force, closed forms or the paper's own
statements (no function is "parity unpinned").
"""
from .ppd_oracle import *  # noqa: F401,F403
