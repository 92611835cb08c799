"""CPU oracle for RMM -- test infrastructure only (see ``rmm_oracle``).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product path never does.
"""
from .rmm_oracle import *  # noqa: F401,F403
from .rmm_oracle import __all__  # noqa: F401
