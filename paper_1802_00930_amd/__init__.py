"""MI355X-native Dynamic Fixed Point (DFP) INT16 convolution.

Das et al., "Mixed Precision Training of Convolutional Neural Networks using
Integer Operations" (ICLR 2018): shared-exponent INT16 quantisation, chunked
INT16 x INT16 -> INT32 convolutions (forward, backward-data, backward-weights)
with per-chunk INT32 -> FP32 conversion, and max-based down-conversion.

The computation lives in the HIP kernels of ``libdfp.so`` behind the C ABI of
``include/dfp.h``; :mod:`.dfp` is its ctypes binding.
"""
from . import dfp  # noqa: F401
from .dfp import (  # noqa: F401
    Desc, DfpError, dfp_conv_bwd_data, dfp_conv_bwd_weights, dfp_conv_fwd, dfp_downconvert, dfp_quantize,
    make_desc, new_scale, read_scale,
)
