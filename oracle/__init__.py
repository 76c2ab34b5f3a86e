"""CPU oracle for carry-through checksum CNN inference: TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the GPU
library (``paper_2609_16742_amd``), and neither imports the other.
"""
from .core import *  # noqa: F401,F403
from .core import build, lib  # noqa: F401
