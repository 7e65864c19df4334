"""GASLoC gossip round on AMD MI355X: Python binding of libgasloc.so.

The compute lives in hand-written HIP kernels behind the C ABI declared in
include/gasloc.h; this package only marshals arguments (see gasloc.py).
"""
from .gasloc import *  # noqa: F401,F403
from .gasloc import GASLoC, GaslocError, library  # noqa: F401
