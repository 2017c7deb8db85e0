"""ctypes binding of the gfx950 quantized-convolution library (libqnn.so).

Argument marshalling only: every computation runs in the library's HIP
kernels.  Device tensors are torch tensors on the current HIP device; work is
enqueued on torch's current stream.  If the library is not built the import
of any entry point raises, there is no fallback.

Tensor conventions follow the C ABI (include/qnn.h): packed NHWC uint8
activations, packed M x kh x kw x C uint8 weights, the lower channel in the
less significant bits, int32 outputs for the raw epilogue.
"""
import ctypes
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
# QNN_LIBRARY names another build of the same sources (the sanitizer test
# loads a host-instrumented build)
LIB_PATH = os.environ.get("QNN_LIBRARY") or os.path.join(HERE, "libqnn.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "qnn.h")

EPI_REQUANT, EPI_THRESH1, EPI_RAW32, EPI_STAIR = 0, 1, 2, 3
# qnn_tile.kernel values (include/qnn.h)
TILE_MFMA16, TILE_MFMA32, TILE_FP4, TILE_IMAGE = 16, 32, 4, 1
_EPI_NAMES = {"requant": EPI_REQUANT, "thresh1": EPI_THRESH1, "raw32": EPI_RAW32, "stair": EPI_STAIR}

STATUS = {
    0: "QNN_OK", 1: "QNN_ERR_NULL", 2: "QNN_ERR_BITS", 3: "QNN_ERR_SHAPE", 4: "QNN_ERR_PARAM",
    5: "QNN_ERR_ALIGN", 6: "QNN_ERR_OVERFLOW", 7: "QNN_ERR_UNSUPPORTED", 8: "QNN_ERR_DEVICE",
    9: "QNN_ERR_LAUNCH",
}


class QnnError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        msg = lib().qnn_status_string(status).decode()
        super().__init__("%s: %s (%s)" % (where, STATUS.get(status, status), msg))


class Tensor(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("h", ctypes.c_int32), ("w", ctypes.c_int32),
                ("c", ctypes.c_int32), ("bits", ctypes.c_int32)]


class ConvGeom(ctypes.Structure):
    _fields_ = [("kh", ctypes.c_int32), ("kw", ctypes.c_int32), ("stride_h", ctypes.c_int32),
                ("stride_w", ctypes.c_int32), ("pad_h", ctypes.c_int32), ("pad_w", ctypes.c_int32)]


class Tile(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_int32), ("tile_m", ctypes.c_int32), ("tile_n", ctypes.c_int32),
                ("waves", ctypes.c_int32)]


class Epi(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("bias", ctypes.c_void_p), ("mult", ctypes.c_void_p),
                ("shift", ctypes.c_void_p), ("thresh", ctypes.c_void_p),
                ("clip_lo", ctypes.c_int32), ("clip_hi", ctypes.c_int32)]


_lib = None


def lib():
    """Load libqnn.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libqnn.so is not built (run __graft_entry__.build()); "
                               "there is no CPU fallback")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        TP = ctypes.POINTER(Tensor)
        L.qnn_abi_version.restype = ctypes.c_int32
        L.qnn_abi_version.argtypes = []
        L.qnn_status_string.restype = ctypes.c_char_p
        L.qnn_status_string.argtypes = [ctypes.c_int]
        L.qnn_device_check.restype = ctypes.c_int
        L.qnn_device_check.argtypes = []
        L.qnn_pixel_bytes.restype = ctypes.c_size_t
        L.qnn_pixel_bytes.argtypes = [TP]
        L.qnn_tensor_bytes.restype = ctypes.c_size_t
        L.qnn_tensor_bytes.argtypes = [TP]
        L.qnn_conv2d_out_shape.restype = ctypes.c_int
        L.qnn_conv2d_out_shape.argtypes = [TP, ctypes.c_int32, ctypes.POINTER(ConvGeom),
                                           ctypes.c_int32, TP]
        L.qnn_conv2d.restype = ctypes.c_int
        L.qnn_conv2d.argtypes = [TP, P, ctypes.c_int32, P, ctypes.POINTER(ConvGeom),
                                 ctypes.POINTER(Epi), TP, P, P]
        L.qnn_conv2d_tiled.restype = ctypes.c_int
        L.qnn_conv2d_tiled.argtypes = [TP, P, ctypes.c_int32, P, ctypes.POINTER(ConvGeom),
                                       ctypes.POINTER(Epi), ctypes.POINTER(Tile), TP, P, P]
        L.qnn_conv2d_maxpool.restype = ctypes.c_int
        L.qnn_conv2d_maxpool.argtypes = [TP, P, ctypes.c_int32, P, ctypes.POINTER(ConvGeom),
                                         ctypes.POINTER(Epi), ctypes.c_int32, ctypes.c_int32, TP, P, P]
        L.qnn_linear.restype = ctypes.c_int
        L.qnn_linear.argtypes = [TP, P, ctypes.c_int32, P, ctypes.POINTER(Epi), TP, P, P]
        L.qnn_maxpool2d.restype = ctypes.c_int
        L.qnn_maxpool2d.argtypes = [TP, P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_int32, TP, P, P]
        L.qnn_relu_s8.restype = ctypes.c_int
        L.qnn_relu_s8.argtypes = [P, P, ctypes.c_size_t, P]
        L.qnn_pack_host.restype = ctypes.c_int
        L.qnn_pack_host.argtypes = [P, ctypes.c_size_t, ctypes.c_int32, P]
        L.qnn_unpack_host.restype = ctypes.c_int
        L.qnn_unpack_host.argtypes = [P, ctypes.c_size_t, ctypes.c_int32, ctypes.c_int32, P]
        _lib = L
    return _lib


def header_functions():
    """Names of the functions include/qnn.h declares."""
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(qnn_[a-z0-9_]+)\s*\(", text)))


def _check(status, where):
    if status != 0:
        raise QnnError(status, where)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _epi(kind, bias, mult, shift, thresh, clip):
    if isinstance(kind, str):
        kind = _EPI_NAMES[kind]
    return Epi(kind, _ptr(bias).value if bias is not None else None,
               _ptr(mult).value if mult is not None else None,
               _ptr(shift).value if shift is not None else None,
               _ptr(thresh).value if thresh is not None else None, clip[0], clip[1]), kind


def pixel_bytes(c, bits):
    return 4 * c if bits == 32 else (c * bits + 7) // 8


def out_shape(xshape, bits, m, kh, kw, stride=(1, 1), pad=(0, 0), epi="requant"):
    """(n, ho, wo, m, out_bits) of a convolution, computed by the library."""
    kind = _EPI_NAMES[epi] if isinstance(epi, str) else epi
    x = Tensor(*xshape, bits)
    y = Tensor()
    _check(lib().qnn_conv2d_out_shape(ctypes.byref(x), m, ctypes.byref(ConvGeom(kh, kw, *stride, *pad)),
                                      kind, ctypes.byref(y)), "qnn_conv2d_out_shape")
    return (y.n, y.h, y.w, y.c, y.bits)


def _out_tensor(shape, out, device):
    import torch
    n, h, w, c, bits = shape
    if bits == 32:
        want = (n, h, w, c)
        dtype = torch.int32
    else:
        want = (n, h, w, pixel_bytes(c, bits))
        dtype = torch.uint8
    if out is None:
        return torch.empty(want, dtype=dtype, device=device)
    if tuple(out.shape) != want or out.dtype != dtype or not out.is_contiguous():
        raise ValueError("out must be a contiguous %s tensor of shape %s" % (dtype, want))
    return out


def conv2d(x, xshape, bits, w, m, kh, kw, stride=(1, 1), pad=(0, 0), epi="requant", bias=None,
           mult=None, shift=None, thresh=None, clip=(0, 0), out=None, stream=None, tile=None):
    """Quantized convolution (qnn_conv2d).  x: uint8 packed NHWC device tensor
    of logical shape xshape = (n, h, w, c); w: uint8 packed weights.  Returns
    uint8 [N, Ho, Wo, out bytes] codes or int32 [N, Ho, Wo, M] (raw32).
    tile = (kernel, tile_m, tile_n, waves) picks the tile shape
    (qnn_conv2d_tiled) instead of the library."""
    yshape = out_shape(xshape, bits, m, kh, kw, stride, pad, epi)
    y = _out_tensor(yshape, out, x.device)
    e, _ = _epi(epi, bias, mult, shift, thresh, clip)
    xd = Tensor(*xshape, bits)
    yd = Tensor(*yshape)
    g = ConvGeom(kh, kw, stride[0], stride[1], pad[0], pad[1])
    if tile is None:
        _check(lib().qnn_conv2d(ctypes.byref(xd), _ptr(x), m, _ptr(w), ctypes.byref(g),
                                ctypes.byref(e), ctypes.byref(yd), _ptr(y), _stream(stream)), "qnn_conv2d")
    else:
        t = Tile(*tile)
        _check(lib().qnn_conv2d_tiled(ctypes.byref(xd), _ptr(x), m, _ptr(w), ctypes.byref(g),
                                      ctypes.byref(e), ctypes.byref(t), ctypes.byref(yd), _ptr(y),
                                      _stream(stream)), "qnn_conv2d_tiled")
    return y


def conv2d_maxpool(x, xshape, bits, w, m, kh, kw, stride=(1, 1), pad=(0, 0), epi="requant",
                   bias=None, mult=None, shift=None, thresh=None, clip=(0, 0), out=None, stream=None):
    """Convolution fused with 2x2 / stride-2 max-pooling (qnn_conv2d_maxpool).
    Returns uint8 [N, floor(Ho/2), floor(Wo/2), out bytes] codes."""
    n, ho, wo, c, obits = out_shape(xshape, bits, m, kh, kw, stride, pad, epi)
    yshape = (n, ho // 2, wo // 2, c, obits)
    y = _out_tensor(yshape, out, x.device)
    e, _ = _epi(epi, bias, mult, shift, thresh, clip)
    xd = Tensor(*xshape, bits)
    yd = Tensor(*yshape)
    g = ConvGeom(kh, kw, stride[0], stride[1], pad[0], pad[1])
    _check(lib().qnn_conv2d_maxpool(ctypes.byref(xd), _ptr(x), m, _ptr(w), ctypes.byref(g),
                                    ctypes.byref(e), 2, 2, ctypes.byref(yd), _ptr(y), _stream(stream)),
           "qnn_conv2d_maxpool")
    return y


def linear(x, xshape, bits, w, m, epi="raw32", bias=None, mult=None, shift=None, thresh=None,
           clip=(0, 0), out=None, stream=None):
    """Fully connected layer (qnn_linear) over the whole NHWC image."""
    kind = _EPI_NAMES[epi] if isinstance(epi, str) else epi
    obits = {EPI_REQUANT: bits, EPI_THRESH1: 1, EPI_RAW32: 32}[kind]
    yshape = (xshape[0], 1, 1, m, obits)
    y = _out_tensor(yshape, out, x.device)
    e, _ = _epi(kind, bias, mult, shift, thresh, clip)
    xd = Tensor(*xshape, bits)
    yd = Tensor(*yshape)
    _check(lib().qnn_linear(ctypes.byref(xd), _ptr(x), m, _ptr(w), ctypes.byref(e),
                            ctypes.byref(yd), _ptr(y), _stream(stream)), "qnn_linear")
    return y


def maxpool2d(x, xshape, bits, kh, kw, sh, sw, out=None, stream=None):
    """Max-pooling over packed unsigned codes (qnn_maxpool2d)."""
    n, h, w_, c = xshape
    ho = (h - kh) // sh + 1
    wo = (w_ - kw) // sw + 1
    yshape = (n, ho, wo, c, bits)
    y = _out_tensor(yshape, out, x.device)
    xd = Tensor(*xshape, bits)
    yd = Tensor(*yshape)
    _check(lib().qnn_maxpool2d(ctypes.byref(xd), _ptr(x), kh, kw, sh, sw, ctypes.byref(yd),
                               _ptr(y), _stream(stream)), "qnn_maxpool2d")
    return y


def relu_s8(x, out=None, stream=None):
    """Signed 8-bit ReLU (qnn_relu_s8); out may be x (in place)."""
    import torch
    y = torch.empty_like(x) if out is None else out
    _check(lib().qnn_relu_s8(_ptr(x), _ptr(y), x.numel(), _stream(stream)), "qnn_relu_s8")
    return y


def device_check():
    _check(lib().qnn_device_check(), "qnn_device_check")


def pack_host(codes, bits):
    """Host packing of unsigned codes (numpy uint8 array) -> packed bytes."""
    import numpy as np
    codes = np.ascontiguousarray(codes, dtype=np.uint8).reshape(-1)
    out = np.zeros((codes.size * bits + 7) // 8, dtype=np.uint8)
    _check(lib().qnn_pack_host(codes.ctypes.data_as(ctypes.c_void_p), codes.size, bits,
                               out.ctypes.data_as(ctypes.c_void_p)), "qnn_pack_host")
    return out


def unpack_host(packed, count, bits, signed):
    import numpy as np
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    out = np.zeros(count, dtype=np.int32)
    _check(lib().qnn_unpack_host(packed.ctypes.data_as(ctypes.c_void_p), count, bits,
                                 1 if signed else 0, out.ctypes.data_as(ctypes.c_void_p)),
           "qnn_unpack_host")
    return out
