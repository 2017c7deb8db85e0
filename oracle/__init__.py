"""CPU oracle for the quantized convolution layer (test infrastructure only).

The arithmetic lives in ``qnn_oracle.c`` (plain C, no intrinsics); this module
only builds it with gcc and marshals numpy arrays.  Only the test suite, the
smoke check and the benchmark's CPU-baseline leg may import it.  It does not
import, and is not imported by, the GPU library.

Citations (paper: Garofalo et al., PULP-NN):
  * Sec. III-A, Eq. (2): integer accumulation of the layer;
  * Sec. III-B, Eq. (6): output = dot(filter bank, im2col column), HWC layout;
  * Sec. III-A: scale-and-clamp compression; Eq. (5): binary XNOR/popcount
    (the oracle uses the equivalent +1/-1 product form);
  * Sec. IV-A: sub-byte storage, fully connected, ReLU and max-pooling.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "qnn_oracle.c")
# QNN_ORACLE_LIB names another build of the same source (the sanitizer test
# runs the pins against an ASan/UBSan build)
_LIB = os.environ.get("QNN_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")

REQUANT, THRESH1, RAW32, STAIR = 0, 1, 2, 3

_lib = None


def build(force=False):
    """Compile the oracle with gcc (-O2, no vector intrinsics)."""
    if os.environ.get("QNN_ORACLE_LIB"):
        return _LIB
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
                               "-pthread", _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32 = ctypes.c_int32
        lib.oracle_conv2d.restype = ctypes.c_int
        lib.oracle_conv2d.argtypes = [P, i32, i32, i32, i32, i32, P, i32, i32, i32, i32, i32, i32,
                                      i32, i32, P, P, P, P, i32, i32, P, P, i32]
        lib.oracle_linear.restype = ctypes.c_int
        lib.oracle_linear.argtypes = [P, i32, i32, i32, P, i32, i32, P, P, P, P, i32, i32, P, P]
        lib.oracle_maxpool2d.restype = ctypes.c_int
        lib.oracle_maxpool2d.argtypes = [P, i32, i32, i32, i32, i32, i32, i32, i32, i32, P]
        lib.oracle_relu_s8.restype = None
        lib.oracle_relu_s8.argtypes = [P, ctypes.c_size_t, P]
        lib.oracle_unpack.restype = None
        lib.oracle_unpack.argtypes = [P, ctypes.c_size_t, i32, i32, P]
        lib.oracle_pack.restype = None
        lib.oracle_pack.argtypes = [P, ctypes.c_size_t, i32, P]
        lib.oracle_packed_bytes.restype = ctypes.c_size_t
        lib.oracle_packed_bytes.argtypes = [ctypes.c_size_t, i32]
        lib.oracle_out_dim.restype = i32
        lib.oracle_out_dim.argtypes = [i32, i32, i32, i32]
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def packed_bytes(count, bits):
    return int(_load().oracle_packed_bytes(count, bits))


def out_dim(size, k, stride, pad):
    return int(_load().oracle_out_dim(size, k, stride, pad))


def unpack(packed, count, bits, signed):
    """Decode `count` codes; values are unsigned/two's complement, or +-1 at 1 bit."""
    packed = _c(packed, np.uint8)
    out = np.empty(count, dtype=np.int32)
    _load().oracle_unpack(_ptr(packed), count, bits, 1 if signed else 0, _ptr(out))
    return out


def pack(codes, bits):
    codes = _c(codes, np.uint32).reshape(-1)
    out = np.empty(packed_bytes(codes.size, bits), dtype=np.uint8)
    _load().oracle_pack(_ptr(codes), codes.size, bits, _ptr(out))
    return out


def _epi_arrays(m, bias, mult, shift, thresh):
    return (_c(bias, np.int32), _c(mult, np.int32), _c(shift, np.int8), _c(thresh, np.int32))


def conv2d(x, shape, bits, w, m, kh, kw, stride=(1, 1), pad=(0, 0), epi=RAW32, bias=None,
           mult=None, shift=None, thresh=None, clip=(0, 0), want_acc=False, want_y=True,
           nthreads=1):
    """Quantized convolution on packed NHWC bytes.

    x: uint8 packed input, shape (N, H, W, Pb) or flat; shape = (N, H, W, C).
    w: uint8 packed OHWI weights.  Returns (acc int64 [N,Ho,Wo,M] or None,
    y uint8 [N,Ho,Wo,Yb] / int32 [N,Ho,Wo,M] or None).
    """
    n, h, wd, c = shape
    ho, wo = out_dim(h, kh, stride[0], pad[0]), out_dim(wd, kw, stride[1], pad[1])
    x = _c(x, np.uint8)
    w = _c(w, np.uint8)
    b, mu, sh, th = _epi_arrays(m, bias, mult, shift, thresh)
    acc = np.zeros((n, ho, wo, m), dtype=np.int64) if want_acc else None
    y = None
    if want_y:
        if epi == RAW32:
            y = np.zeros((n, ho, wo, m), dtype=np.int32)
        else:
            obits = bits if epi in (REQUANT, STAIR) else 1
            y = np.zeros((n, ho, wo, packed_bytes(m, obits)), dtype=np.uint8)
    rc = _load().oracle_conv2d(_ptr(x), n, h, wd, c, bits, _ptr(w), m, kh, kw, stride[0],
                               stride[1], pad[0], pad[1], epi, _ptr(b), _ptr(mu), _ptr(sh),
                               _ptr(th), clip[0], clip[1], _ptr(acc), _ptr(y), nthreads)
    if rc != 0:
        raise ValueError("oracle_conv2d rejected its arguments")
    return acc, y


def linear(x, n, k, bits, w, m, epi=RAW32, bias=None, mult=None, shift=None, thresh=None,
           clip=(0, 0), want_acc=False):
    x = _c(x, np.uint8)
    w = _c(w, np.uint8)
    b, mu, sh, th = _epi_arrays(m, bias, mult, shift, thresh)
    acc = np.zeros((n, m), dtype=np.int64) if want_acc else None
    if epi == RAW32:
        y = np.zeros((n, m), dtype=np.int32)
    else:
        y = np.zeros((n, packed_bytes(m, bits if epi in (REQUANT, STAIR) else 1)), dtype=np.uint8)
    rc = _load().oracle_linear(_ptr(x), n, k, bits, _ptr(w), m, epi, _ptr(b), _ptr(mu), _ptr(sh),
                               _ptr(th), clip[0], clip[1], _ptr(acc), _ptr(y))
    if rc != 0:
        raise ValueError("oracle_linear rejected its arguments")
    return acc, y


def maxpool2d(x, shape, bits, kh, kw, sh, sw):
    n, h, w, c = shape
    ho, wo = out_dim(h, kh, sh, 0), out_dim(w, kw, sw, 0)
    x = _c(x, np.uint8)
    y = np.zeros((n, ho, wo, packed_bytes(c, bits)), dtype=np.uint8)
    rc = _load().oracle_maxpool2d(_ptr(x), n, h, w, c, bits, kh, kw, sh, sw, _ptr(y))
    if rc != 0:
        raise ValueError("oracle_maxpool2d rejected its arguments")
    return y


def relu_s8(x):
    x = _c(x, np.int8)
    y = np.empty_like(x)
    _load().oracle_relu_s8(_ptr(x), x.size, _ptr(y))
    return y
