"""MI355X-native expand / FIFO batch / ordered gather core (RayOrch's
lineage-controlled dataflow, arXiv 2609.18703).

The compute path is ``libro.so`` (hand-written HIP for gfx950) behind the C
ABI in ``include/ro.h``; :mod:`.ro` is its Python binding.
"""
from .ro import *  # noqa: F401,F403
