"""MI355X-native Blockwise Parallel Transformer layer (libbpt) and its Python binding.

The compute path is the HIP library ``libbpt.so`` built from ``csrc/`` for gfx950;
``bpt`` is a ctypes binding that only marshals arguments.
"""
from . import bpt  # noqa: F401
