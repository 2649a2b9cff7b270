"""NEURON-Fabric bucket reducer for AMD MI355X (gfx950).

The product is the HIP library libnf.so with the C ABI declared in
include/nf.h; `binding` is its ctypes binding with the same function names.
"""
from .binding import *  # noqa: F401,F403
from .binding import load, EXPORTS, NFError  # noqa: F401
