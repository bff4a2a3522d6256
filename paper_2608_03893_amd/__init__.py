"""MI355X-native cross-model KV cache mapper.

The product is the C-ABI library ``libkvx.so`` (HIP kernels for gfx950, see
``include/kvx.h``); ``paper_2608_03893_amd.kvx`` is its thin ctypes binding.
Importing this package loads nothing; import ``paper_2608_03893_amd.kvx`` to
load the library.
"""

__version__ = "0.1.0"
