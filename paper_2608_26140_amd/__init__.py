"""MI355X-native selective affix-KV recompute (ACache hot path).

The compute lives in libacache.so (hand-written gfx950 HIP kernels behind a
C ABI, include/acache.h).  `paper_2608_26140_amd.acache` is the ctypes
binding; `paper_2608_26140_amd.driver` sequences the calls for a stack.
Importing the binding raises ImportError when the library is not built.
"""

__version__ = "0.1.0"
