"""Seeded synthetic workloads shared by the CPU oracle and the GPU library.

Holds architecture descriptors and random-number recipes only; none of the
carry-through method's arithmetic lives in this package.
"""
from .nets import Net, CONFIGS, config, by_name  # noqa: F401
from . import gen  # noqa: F401
