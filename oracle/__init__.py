"""fp64 CPU oracle of the SCD KV-state codec (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline leg may import
this package.  The product path never does.
"""
from .scd_oracle import *  # noqa: F401,F403
from . import scd_oracle  # noqa: F401
