"""LibraSpec verification hot path for AMD MI355X (gfx950).

``lsv`` is the ctypes binding of liblsv.so (C-ABI in include/lsv.h);
``runtime`` allocates device buffers with torch and packs weights.
"""
from . import lsv  # noqa: F401
