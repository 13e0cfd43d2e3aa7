"""MI355X-native storage-side feature extraction for split transfer learning.

Runs the frozen-layer forward pass of a CNN or ViT feature extractor from the
input images up to a split layer, plus the per-layer output-size and time
profile used to choose the split (the storage-side hot path of HAPI,
Petrescu et al.).  All compute runs in the HIP kernels of ``libhapi.so``
(gfx950); this package is the ctypes binding (``binding``) and the layer
descriptors of the evaluated models (``models``).
"""
from .binding import *  # noqa: F401,F403
from .binding import Desc, HapiError  # noqa: F401
from . import models  # noqa: F401
