"""MI355X-native Action-Subspace-Protected (ASP) W4A4 linear layer of Q-WAM.

The compute lives in libqwam.so (hand-written HIP kernels for gfx950 behind a
C ABI, include/qwam.h).  `qwam` is its thin ctypes binding, `calib` builds a
layer's factors offline, `inputs` draws the seeded synthetic workloads.
"""
from .qwam import (PackedLayer, QwamError, asp_linear, debug_group_partials, forward,  # noqa: F401
                   lib, make_layer, pack_weights, quantize_act)

__all__ = ["PackedLayer", "QwamError", "asp_linear", "debug_group_partials", "forward", "lib",
           "make_layer", "pack_weights", "quantize_act"]
