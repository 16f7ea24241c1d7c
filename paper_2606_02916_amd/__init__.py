"""MI355X-native per-window feature-fetch path of GreenGNN (arXiv 2606.02916).

``gg`` is the ctypes binding of libgg.so (include/gg.h); ``window`` holds the
buffer sets and call sequences of the sequential and look-ahead drivers;
``sage`` runs the GraphSAGE consumer of the gathered rows.  Importing the
package loads the HIP library and fails loudly if it is not built.
"""
from . import gg  # noqa: F401
from .sage import SageConsumer  # noqa: F401
from .window import FetchPipeline, LookaheadPipeline  # noqa: F401
