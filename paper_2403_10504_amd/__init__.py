"""MI355X-native swapped GPT training step (Atom, arXiv 2403.10504).

The product is libatom.so (C ABI in include/atom.h, kernels for gfx950);
`atom` is its ctypes binding and `Session` wires it to a PyTorch device
arena and streams.
"""
from . import atom  # noqa: F401
from .session import Session  # noqa: F401
