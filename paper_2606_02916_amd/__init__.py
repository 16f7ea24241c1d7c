"""MI355X-native per-window feature-fetch path of GreenGNN (arXiv 2606.02916).

``gg`` is the ctypes binding of libgg.so (include/gg.h); ``window`` holds the
buffer set and call sequence of one window.  Importing the package loads the
HIP library and fails loudly if it is not built.
"""
from . import gg  # noqa: F401
from .window import FetchPipeline, LookaheadPipeline  # noqa: F401
