"""Seeded synthetic workloads shared by the tests, ``bench.py`` and ``smoke()``.

This package holds the input recipe only (shapes, role-label patterns, random
Q/K/V and the sink-bias construction).  It contains none of the method's
arithmetic: no softmax, no score, no pooling, no allocation, no selection.
Both the HIP library and the CPU oracle receive the very same tensors it
produces.
"""

from .gen import *  # noqa: F401,F403
