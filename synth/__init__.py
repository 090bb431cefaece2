"""Seeded synthetic inputs shared by the oracle tests, the GPU parity tests and the benchmark.

Holds no arithmetic of the codec itself.
"""
from .workloads import *  # noqa: F401,F403
from . import workloads  # noqa: F401
