"""CPU oracle for the ShiftQuant backward path.  TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never does, and it
shares no code with the HIP path.
"""
from .oracle import *  # noqa: F401,F403
