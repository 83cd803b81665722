"""MI355X (gfx950) implementation of TransAct V2's lifelong-sequence serving
hot path: candidate-anchored NN select over the de-duplicated request-level
sequence, token gather and the fused-candidate causal encoder.

The compute lives in libtav2.so (HIP kernels behind the C ABI of
include/tav2.h); `paper_2506_02267_amd.tav2` is its thin Python binding.
"""
from . import tav2  # noqa: F401
from .tav2 import (DeviceCands, DeviceSeq, DeviceTokens, DeviceWeights, SelectEncode,  # noqa: F401
                   Workspace, encode, gather, load_library, nn_select, select_encode)
