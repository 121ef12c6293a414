"""CPU oracle for Looped Latent Attention -- test infrastructure only.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
import this package.  It shares no code with the HIP library.
"""
from .lla_oracle import *  # noqa: F401,F403
from .lla_oracle import __all__  # noqa: F401
