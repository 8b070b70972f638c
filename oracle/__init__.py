"""CPU oracle for the MuonBP optimizer step.

Test infrastructure: only tests, the smoke check and the benchmark's
CPU-baseline leg may import it.  The product path never does.
"""
from .muonbp_oracle import *  # noqa: F401,F403
