"""CPU oracle for the block-routed MoE layer (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never calls it and
shares no code with it.
"""
from .dmoe_oracle import *  # noqa: F401,F403
