"""fp64 CPU oracle of the xPress refine + verify path.

TEST INFRASTRUCTURE: imported only by tests/, by __graft_entry__.smoke() and by
the CPU-baseline leg of bench.py.  The device path (paper_2608_02438_amd) never
imports it and shares no code with it.
"""
from .xpress_ref import *  # noqa: F401,F403
from . import layer_ref  # noqa: F401,E402  (the context layer)
