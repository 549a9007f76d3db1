"""CPU oracle for the CAT W4A4 linear-layer path -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU
baseline leg may import this package.  The product path never does.
"""
from . import cat_oracle  # noqa: F401
from .cat_oracle import *  # noqa: F401,F403
