"""fp64 CPU oracle of the CacheRepair repair forward pass (test infrastructure).

Only the test suite, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may import this package.  The product path never does.
"""
from .repair import *  # noqa: F401,F403
from .repair import __all__  # noqa: F401
