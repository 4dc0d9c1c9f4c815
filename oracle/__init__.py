"""CPU oracle of the selective-update hot path: test infrastructure only.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
import this package; the product path never does.
"""

from .zf_oracle import *  # noqa: F401,F403
