"""fp64 CPU oracle for the MomentKV hot path.

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the CPU
baseline leg of the benchmark.  Nothing in the product package imports it.
"""
from .momentkv import *  # noqa: F401,F403
from .momentkv import __all__  # noqa: F401
