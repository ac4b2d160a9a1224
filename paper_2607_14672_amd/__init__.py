"""MI355X-native DSTD-LIF layers: HIP kernels behind a C ABI (libdstd_lif.so)."""
from . import dstd  # noqa: F401
from .dstd import (  # noqa: F401
    make_params, make_conv_shape, forward, backward, conv_forward, conv_backward,
    softmax_ce_grad, mse_grad, DSTDError,
)
