"""MI355X (gfx950) tree-verification library for AceSpec's cloud side.

The compute path is the HIP library ``libacespec.so`` (sources in ``csrc/``, C ABI in
``include/acespec.h``); ``acespec`` is its ctypes binding.
"""
from . import acespec  # noqa: F401
