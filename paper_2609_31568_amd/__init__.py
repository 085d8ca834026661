"""MI355X (gfx950) cluster-level sparse prefill: the hot path of Similarity Chunk Rolling.

The computation lives in libscale.so (hand-written HIP kernels behind the C ABI of
include/scale.h); this package is its ctypes binding plus a per-layer driver.
"""
from .binding import *  # noqa: F401,F403
from .binding import (EXPORTS, STAGES, Config, Scale, ScaleError, make_config, scale_config,  # noqa: F401
                      scale_variant, status_string)
from .pipeline import LayerBuffers, config_for, run_layer  # noqa: F401
