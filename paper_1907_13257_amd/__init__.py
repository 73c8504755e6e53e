"""liblstm355: the per-worker training step (forward + BPTT) of stacked
LSTM / LSTMP layers as hand-written HIP kernels for the MI355X (gfx950).

`lstm355` is the ctypes binding of the C ABI declared in include/lstm355.h;
`build` compiles the shared library in-tree.  The library is loaded on first
use and its absence is an error: there is no fallback path.
"""
from . import lstm355  # noqa: F401
from .lstm355 import Layer, Stack, StackLayer, load_library  # noqa: F401
