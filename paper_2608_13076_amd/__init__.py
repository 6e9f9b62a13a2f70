"""MI355X-native speculative-verify path (SPADE, arXiv 2608.13076).

The compute lives in ``libspade.so`` (HIP for gfx950, C ABI in
``include/spade.h``); ``spade`` is its ctypes binding.  Import
``paper_2608_13076_amd.spade`` to use it.
"""

__all__ = ["spade", "build"]
