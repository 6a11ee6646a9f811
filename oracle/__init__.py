"""CPU oracle for the OasisKV decode path (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.
"""
from .oasis_oracle import *  # noqa: F401,F403
