"""CPU oracle (TEST INFRASTRUCTURE): plain NumPy definitions of the
error-feedback compressors and the aggregate.  Imported only by tests/,
__graft_entry__.smoke() and bench.py's CPU-baseline leg."""

from . import efsparse_oracle, philox  # noqa: F401
from .efsparse_oracle import *  # noqa: F401,F403
