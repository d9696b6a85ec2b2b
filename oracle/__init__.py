"""CPU oracle for the V-MoE layer (TEST INFRASTRUCTURE ONLY).

Plain, slow, obviously-correct reference used to check the HIP path. Only
`tests/`, `__graft_entry__.smoke()` and the CPU-baseline leg of `bench.py`
may import it; the product package never does. It shares no code with the
HIP library: the arithmetic lives in `vmoe_oracle.c` (plain loops, double
accumulation) and this module only marshals numpy arrays through ctypes.
"""
from .api import *  # noqa: F401,F403
from .api import build, load  # noqa: F401
