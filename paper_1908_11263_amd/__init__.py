"""MI355X (gfx950) quantized convolution layer of PULP-NN: INT-8/4/2/1
convolution with int32 accumulation and fused per-channel compression, plus
fully connected, max-pooling and ReLU helpers, and the convolution fused with
its 2x2 max-pooling, behind a C ABI (include/qnn.h).
"""
from .qnn import (EPI_RAW32, EPI_REQUANT, EPI_STAIR, EPI_THRESH1, TILE_FP4, TILE_MFMA16,  # noqa: F401
                  TILE_MFMA32, TILE_IMAGE, QnnError, conv2d,
                  conv2d_maxpool, device_check, lib, linear, maxpool2d, out_shape, pack_host,
                  pixel_bytes, relu_s8, unpack_host)
