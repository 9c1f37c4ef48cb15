"""MI355X (gfx950) implementation of PETRA's per-stage reversible step.

The compute path is libpetra.so (hand-written HIP kernels behind the C ABI
of include/petra.h); this package holds its ctypes binding and a small
buffer-owning helper.  Importing the package loads the library and fails if
it has not been built.
"""
from . import _lib
from ._lib import *  # noqa: F401,F403  (the petra_* wrappers, same names as the C ABI)

_lib.load()

from .stage import Net, Stage, to_host  # noqa: E402,F401
