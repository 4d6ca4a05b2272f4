"""fp64 CPU oracle of the DP-SGD ghost-clipping hot path (test infrastructure).

Only the test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. The GPU library never does.
"""
from .dp_oracle import *  # noqa: F401,F403
from .dp_oracle import __all__  # noqa: F401
