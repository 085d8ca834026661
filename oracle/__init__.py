"""fp64 CPU oracle for cluster-level sparse prefill -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may use it.
It shares no code with the HIP path and never imports it.
"""
from .scr import *  # noqa: F401,F403
from .scr import __all__  # noqa: F401
