"""CPU oracle for the UniQuan_F fake-quant step.

TEST INFRASTRUCTURE ONLY: imported by tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py, never by the library or its binding.
"""
from . import uniquan  # noqa: F401
from .uniquan import *  # noqa: F401,F403
