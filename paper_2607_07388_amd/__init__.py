"""TF-Engram phrase-memory lookup + inject for AMD MI355X (gfx950).

The work happens in ``libtfe.so`` (hand-written HIP kernels behind the C ABI
of ``include/tfe.h``); ``tfe`` is its ctypes binding with the same names.
"""
from . import tfe  # noqa: F401
