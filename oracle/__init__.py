"""fp64 CPU oracle of one pipeline stage's stateful decode/verify forward.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
link this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library and is deliberately plain and slow.
"""
from .stage_oracle import *  # noqa: F401,F403
