"""Plain fp64 CPU oracle for the single-GPU Muon step (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP path.
"""
from .muon_ref import *  # noqa: F401,F403
