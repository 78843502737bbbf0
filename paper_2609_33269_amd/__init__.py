"""MI355X-native Action-Subspace-Protected (ASP) W4A4 linear layer of Q-WAM.

The compute lives in libqwam.so (hand-written HIP kernels for gfx950 behind a
C ABI, include/qwam.h).  `qwam` is its thin ctypes binding, `calib` builds a
layer's factors offline, `inputs` draws the seeded synthetic workloads.
"""
from .qwam import (PackedLayer, QwamError, aog_accumulate, aog_protected_basis,  # noqa: F401
                   aog_protected_basis_workspace, asp_layer, asp_linear, debug_group_partials, forward, lib,
                   make_layer, pack_weights, quantize_act, quantize_act_deflated)

__all__ = ["PackedLayer", "QwamError", "aog_accumulate", "aog_protected_basis", "aog_protected_basis_workspace",
           "asp_layer", "asp_linear", "debug_group_partials", "forward", "lib", "make_layer", "pack_weights",
           "quantize_act", "quantize_act_deflated"]
