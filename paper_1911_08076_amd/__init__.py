"""MI355X-native integrated fixed-point quantized convolution (IFQ-Net).

The path: +-1 weights convolved with k-bit activation codes into int32 sums on
int8 MFMA (Eq. 1), conv + BN + quantizer folded into per-channel integer
thresholds (Sec. 3.2, Eq. 6-8) applied in the conv epilogue, integer max-pool
on codes (Eq. 4), and a layer-chain driver. All of it lives in libifq.so
(HIP for gfx950 plus host C++); this package is its Python binding.

Importing the package loads libifq.so and raises ImportError if it has not
been built: there is no CPU fallback.
"""
from . import _ffi

_ffi.load()

from .api import *  # noqa: E402,F401,F403
from .api import IfqError  # noqa: E402,F401
from .stack import DeviceStack, conv_ops  # noqa: E402,F401
from ._ffi import (IFQ_LAYOUT_I8_NHWC, IFQ_LAYOUT_U2_NHWC_PACKED,  # noqa: E402,F401
                   IFQ_LAYOUT_I32_NHWC, IFQ_LAYOUT_U2_BLOCK64, IFQ_POOL_VALID, IFQ_POOL_SAME,
                   IFQ_JOIN_NONE, IFQ_JOIN_IDENTITY, IFQ_JOIN_CONV,
                   IFQ_JOIN_CONV_FUSED,
                   IFQ_LAYER_CONV, IFQ_LAYER_POOL, IFQ_LAYER_CONV_POOL,
                   IFQ_LAYER_CONV_FP4, IFQ_LAYER_CONV_POOL_FP4)
