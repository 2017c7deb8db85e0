"""MI355X (gfx950) quantized convolution layer of PULP-NN: INT-8/4/2/1
convolution with int32 accumulation and fused per-channel compression, plus
fully connected, max-pooling and ReLU helpers, behind a C ABI (include/qnn.h).
"""
from .qnn import (EPI_RAW32, EPI_REQUANT, EPI_THRESH1, QnnError, conv2d, device_check,  # noqa: F401
                  lib, linear, maxpool2d, out_shape, pack_host, pixel_bytes, relu_s8, unpack_host)
