"""fp64 CPU oracle for the FrameFT adapter path -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path never does.
"""
from .frameft_oracle import *  # noqa: F401,F403
from .frameft_oracle import NotATightFusionFrame  # noqa: F401
