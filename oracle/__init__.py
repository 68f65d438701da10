"""fp64 CPU oracle of the EOGP hot path (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package; the product path never does.
"""
from .eogp_oracle import *  # noqa: F401,F403
