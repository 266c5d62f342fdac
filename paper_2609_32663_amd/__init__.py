"""Distance-KV inference hot path on MI355X (gfx950).

The work runs in libdkv.so (hand-written HIP kernels behind the C ABI of
include/dkv.h); this package holds the kernel sources (csrc/), the in-tree
build (build.py) and a ctypes binding with the same entry-point names
(binding.py).  Importing the package loads the library and fails loudly if it
has not been built.
"""

from .binding import *  # noqa: F401,F403
from .binding import __all__  # noqa: F401
from .binding import library as _library

_library()
