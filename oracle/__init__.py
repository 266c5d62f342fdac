"""CPU oracle for the Distance-KV hot path (test infrastructure only).

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import this package.  See `dkv_oracle` for what it computes.
"""

from .dkv_oracle import *  # noqa: F401,F403
from .dkv_oracle import __all__  # noqa: F401
