"""MI355X (gfx950) implementation of PETRA's per-stage reversible step.

The compute path is libpetra.so (hand-written HIP kernels behind the C ABI
of include/petra.h); this package holds its ctypes binding and a small
buffer-owning helper.  Importing the package loads the library and fails if
it has not been built.
"""
# torch first: it ships its own HIP runtime under the same soname as the
# system one, and the library must bind to the runtime that owns the device
# memory torch hands it
import torch  # noqa: F401,E402

from . import _lib  # noqa: E402
from ._lib import *  # noqa: F401,F403,E402  (the petra_* wrappers, same names as the C ABI)

_lib.load()

from .stage import Net, Stage, to_host  # noqa: E402,F401
