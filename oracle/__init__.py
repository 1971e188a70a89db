"""float64 CPU oracle of the RKSC verify pass (test infrastructure only).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this package; the HIP product path never does.
"""
from .rksc_oracle import *  # noqa: F401,F403
from .rksc_oracle import __all__  # noqa: F401
