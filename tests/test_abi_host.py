"""C-ABI checks that need no GPU: the library loads, exports every function
its header declares, validates arguments on the host (before any device
call) and its host packing helpers agree with the generator and the oracle."""
import ctypes

import numpy as np
import pytest

import synth


@pytest.fixture(scope="module")
def q():
    import paper_1908_11263_amd as q
    return q


@pytest.fixture(scope="module")
def L(q):
    return q.lib()


def test_exports_every_header_function(q, L):
    names = q.qnn.header_functions()
    assert len(names) >= 12
    for name in names:
        assert hasattr(L, name), name
    assert L.qnn_abi_version() == 8


def test_exports_every_calibration_function(q, L):
    """The measurement entry points (include/qnn_calib.h) are exported and
    refuse bad arguments on the host, before any device call."""
    import os
    import re
    path = os.path.join(os.path.dirname(q.qnn.HEADER), "qnn_calib.h")
    with open(path) as f:
        text = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(qnn_calib_[a-z0-9_]+)\s*\(", text)))
    assert names == ["qnn_calib_copy", "qnn_calib_empty", "qnn_calib_mfma_i8", "qnn_calib_xnor"]
    for name in names:
        assert hasattr(L, name), name
    P, i32 = ctypes.c_void_p, ctypes.c_int32
    for name in ("qnn_calib_mfma_i8", "qnn_calib_xnor"):
        f = getattr(L, name)
        f.restype = ctypes.c_int
        f.argtypes = [i32, i32, P, P, P]
        assert f(4, 10, None, None, None) == 1                 # NULL output
        assert f(0, 10, P(4096), None, None) == 4              # no workgroups
        assert f(1 << 21, 10, P(4096), None, None) == 4        # too many
        assert f(4, 0, P(4096), None, None) == 4               # no iterations
        assert f(4, 10, P(4100), None, None) == 5              # misaligned output
        assert f(4, 10, P(4096), P(4104), None) == 5           # misaligned clock buffer
    L.qnn_calib_copy.restype = ctypes.c_int
    L.qnn_calib_copy.argtypes = [P, P, ctypes.c_size_t, P]
    assert L.qnn_calib_copy(None, P(4096), 16, None) == 1
    assert L.qnn_calib_copy(P(4096), P(8192), 17, None) == 5   # not whole quads
    assert L.qnn_calib_copy(P(4096), P(4112), 32, None) == 4   # overlapping
    assert L.qnn_calib_copy(P(4096), P(8192), 1 << 41, None) == 3
    L.qnn_calib_empty.restype = ctypes.c_int
    L.qnn_calib_empty.argtypes = [i32, P]
    assert L.qnn_calib_empty(0, None) == 4


def test_status_strings(q, L):
    for code in range(10):
        assert L.qnn_status_string(code)
    assert L.qnn_status_string(123) == b"unknown status"


def test_pixel_and_tensor_bytes(q, L):
    T = q.qnn.Tensor
    assert L.qnn_pixel_bytes(ctypes.byref(T(1, 1, 1, 64, 4))) == 32
    assert L.qnn_pixel_bytes(ctypes.byref(T(1, 1, 1, 3, 8))) == 3
    assert L.qnn_pixel_bytes(ctypes.byref(T(1, 1, 1, 5, 2))) == 2
    assert L.qnn_pixel_bytes(ctypes.byref(T(1, 1, 1, 10, 32))) == 40
    assert L.qnn_tensor_bytes(ctypes.byref(T(64, 32, 32, 64, 4))) == 64 * 32 * 32 * 32
    assert L.qnn_tensor_bytes(None) == 0


def test_out_shape(q):
    assert q.out_shape((1, 16, 16, 32), 8, 32, 3, 3, (1, 1), (1, 1)) == (1, 16, 16, 32, 8)
    assert q.out_shape((2, 9, 7, 256), 1, 70, 3, 3, (2, 2), (1, 1), "thresh1") == (2, 5, 4, 70, 1)
    assert q.out_shape((4, 4, 4, 64), 8, 10, 4, 4, (1, 1), (0, 0), "raw32") == (4, 1, 1, 10, 32)
    with pytest.raises(q.QnnError) as e:
        q.out_shape((1, 2, 2, 32), 8, 4, 5, 5, (1, 1), (0, 0))
    assert e.value.status == 3


FAKE = 1 << 20  # a 16-byte aligned non-NULL address; never dereferenced


def call_conv(q, L, xs, bits, m, g, epi, ys, xp=FAKE, wp=FAKE, yp=FAKE):
    T, G, E = q.qnn.Tensor, q.qnn.ConvGeom, q.qnn.Epi
    return L.qnn_conv2d(ctypes.byref(T(*xs, bits)), xp, m, wp, ctypes.byref(G(*g)),
                        ctypes.byref(E(*epi)), ctypes.byref(T(*ys)), yp, None)


REQ8 = (0, None, FAKE, FAKE, None, 0, 255)


@pytest.mark.parametrize("case,status", [
    (dict(bits=3), 2),                                    # bits not in {1,2,4,8}
    (dict(xs=(1, 0, 4, 32)), 3),                          # empty image
    (dict(m=0), 3),                                       # no filters
    (dict(g=(0, 3, 1, 1, 1, 1)), 4),                      # kernel 0
    (dict(g=(3, 3, 0, 1, 1, 1)), 4),                      # stride 0
    (dict(g=(3, 3, 1, 1, -1, 1)), 4),                     # negative pad
    (dict(g=(9, 9, 1, 1, 0, 0), ys=(1, 0, 0, 32, 8)), 3),  # kernel larger than padded input
    (dict(ys=(1, 4, 4, 32, 4)), 2),                       # wrong output bit-width
    (dict(ys=(1, 4, 5, 32, 8)), 3),                       # wrong output shape
    (dict(epi=(0, None, None, FAKE, None, 0, 255)), 1),   # REQUANT without multipliers
    (dict(epi=(0, None, FAKE, FAKE, None, 0, 256)), 4),   # clip above 2^bits - 1
    (dict(epi=(0, None, FAKE, FAKE, None, 5, 4)), 4),     # clip_lo > clip_hi
    (dict(epi=(0, None, FAKE, FAKE, None, -1, 4)), 4),    # negative clip_lo
    (dict(epi=(1, None, None, None, FAKE, 0, 0)), 2),     # THRESH1 on 8-bit data
    (dict(epi=(7, None, None, None, None, 0, 0)), 4),     # unknown epilogue
    (dict(xs=(1, 4, 4, 3), ys=(1, 4, 4, 32, 8)), 5),      # 3-byte pixels
    (dict(xp=FAKE + 4), 5),                               # misaligned input pointer
    (dict(yp=FAKE + 8), 5),                               # misaligned output pointer
    (dict(xp=None), 1),                                   # NULL input
    (dict(wp=None), 1),                                   # NULL weights
    (dict(xs=(1, 4, 4, 8192), g=(3, 3, 1, 1, 1, 1)), 6),  # K = 73728 > INT-8 limit
])
def test_conv_validation_on_host(q, L, case, status):
    args = dict(xs=(1, 4, 4, 32), bits=8, m=32, g=(3, 3, 1, 1, 1, 1), epi=REQ8,
                ys=(1, 4, 4, 32, 8))
    args.update(case)
    assert call_conv(q, L, **args) == status


REQ4 = (0, None, FAKE, FAKE, None, 0, 15)


@pytest.mark.parametrize("g,xs,ys", [
    ((3, 3, 2, 2, 1, 1), (1, 8, 8, 4), (1, 4, 4, 32, 4)),     # stride 2: not the whole-image kernel
    ((1, 1, 1, 1, 0, 0), (1, 8, 8, 4), (1, 8, 8, 32, 4)),     # 1x1 filter
    ((3, 3, 1, 1, 1, 1), (1, 8, 40, 4), (1, 8, 40, 32, 4)),   # rows of 40 outputs
])
def test_half_word_pixels_outside_the_image_kernel(q, L, g, xs, ys):
    """2-byte pixels (4 channels at 4 bits) are read by the whole-image kernel
    only; other layers are refused on the host with QNN_ERR_ALIGN."""
    assert call_conv(q, L, xs, 4, 32, g, REQ4, ys) == 5


def test_half_word_pixels_at_other_widths(q, L):
    """2-byte pixels at 8 bits (2 channels) or 2 bits (8 channels) are not
    built: QNN_ERR_ALIGN."""
    assert call_conv(q, L, (1, 8, 8, 2), 8, 32, (3, 3, 1, 1, 1, 1), REQ8, (1, 8, 8, 32, 8)) == 5
    assert call_conv(q, L, (1, 8, 8, 8), 2, 32, (3, 3, 1, 1, 1, 1), (0, None, FAKE, FAKE, None, 0, 3),
                     (1, 8, 8, 32, 2)) == 5


def test_int1_requires_threshold_or_raw(q, L):
    assert call_conv(q, L, (1, 4, 4, 32), 1, 8, (3, 3, 1, 1, 1, 1), (0, None, FAKE, FAKE, None, 0, 1),
                     (1, 4, 4, 8, 1)) == 2
    assert call_conv(q, L, (1, 4, 4, 32), 1, 8, (3, 3, 1, 1, 1, 1), (1, None, None, None, None, 0, 0),
                     (1, 4, 4, 8, 1)) == 1


def test_stair_validation(q, L):
    """The staircase epilogue is defined at 4 and 2 bits and needs thresholds."""
    g = (3, 3, 1, 1, 1, 1)
    st4 = (3, None, None, None, FAKE, 0, 0)
    assert q.out_shape((1, 4, 4, 64), 4, 16, 3, 3, (1, 1), (1, 1), "stair") == (1, 4, 4, 16, 4)
    assert q.out_shape((1, 4, 4, 128), 2, 16, 3, 3, (1, 1), (1, 1), "stair") == (1, 4, 4, 16, 2)
    for bits, c in ((8, 32), (1, 32)):
        with pytest.raises(q.QnnError) as e:
            q.out_shape((1, 4, 4, c), bits, 16, 3, 3, (1, 1), (1, 1), "stair")
        assert e.value.status == 2
    assert call_conv(q, L, (1, 4, 4, 32), 8, 16, g, st4, (1, 4, 4, 16, 8)) == 2
    assert call_conv(q, L, (1, 4, 4, 64), 4, 16, g, (3, None, None, None, None, 0, 0),
                     (1, 4, 4, 16, 4)) == 1
    # a valid call gets past every host check (no GPU here: device error)
    assert call_conv(q, L, (1, 4, 4, 64), 4, 16, g, st4, (1, 4, 4, 16, 4)) == 8
    assert call_conv(q, L, (1, 4, 4, 128), 2, 16, g, st4, (1, 4, 4, 16, 2)) == 8


def call_conv_pool(q, L, xs, bits, m, g, epi, ys, pk=2, ps=2, xp=FAKE, wp=FAKE, yp=FAKE):
    T, G, E = q.qnn.Tensor, q.qnn.ConvGeom, q.qnn.Epi
    return L.qnn_conv2d_maxpool(ctypes.byref(T(*xs, bits)), xp, m, wp, ctypes.byref(G(*g)),
                                ctypes.byref(E(*epi)), pk, ps, ctypes.byref(T(*ys)), yp, None)


def test_conv_maxpool_validation(q, L):
    """Fused conv + 2x2/2 max-pool: host checks."""
    g = (3, 3, 1, 1, 1, 1)
    ok = ((1, 8, 8, 32), 8, 16, g, REQ8, (1, 4, 4, 16, 8))
    assert call_conv_pool(q, L, *ok) == 8                               # valid (no GPU here)
    assert call_conv_pool(q, L, *ok, pk=3) == 4                         # only 2x2 windows
    assert call_conv_pool(q, L, *ok, ps=1) == 4                         # only stride 2
    assert call_conv_pool(q, L, (1, 8, 8, 32), 8, 16, g, (2, None, None, None, None, 0, 0),
                          (1, 4, 4, 16, 32)) == 4                        # RAW32 not pooled
    assert call_conv_pool(q, L, (1, 8, 8, 32), 8, 16, g, REQ8, (1, 8, 8, 16, 8)) == 3   # unpooled shape
    assert call_conv_pool(q, L, (1, 7, 9, 32), 8, 16, g, REQ8, (1, 3, 4, 16, 8)) == 8   # floor sizes
    assert call_conv_pool(q, L, (1, 1, 8, 32), 8, 16, (1, 1, 1, 1, 0, 0), REQ8,
                          (1, 0, 4, 16, 8)) == 3                         # conv output 1 row
    assert call_conv_pool(q, L, (1, 8, 8, 256), 1, 16, g, (1, None, None, None, FAKE, 0, 0),
                          (1, 4, 4, 16, 1)) == 2                         # no INT-1 pooling
    st = (3, None, None, None, FAKE, 0, 0)
    assert call_conv_pool(q, L, (2, 6, 6, 64), 4, 40, g, st, (2, 3, 3, 40, 4)) == 8      # staircase


def call_conv_tiled(q, L, xs, bits, m, g, epi, ys, tile):
    T, G, E = q.qnn.Tensor, q.qnn.ConvGeom, q.qnn.Epi
    return L.qnn_conv2d_tiled(ctypes.byref(T(*xs, bits)), FAKE, m, FAKE, ctypes.byref(G(*g)),
                              ctypes.byref(E(*epi)), ctypes.byref(q.qnn.Tile(*tile)),
                              ctypes.byref(T(*ys)), FAKE, None)


def test_conv_tiled_validation(q, L):
    """Caller-chosen tile shapes: only built shapes are accepted."""
    g = (3, 3, 1, 1, 1, 1)
    args = ((1, 8, 8, 32), 8, 64, g, REQ8, (1, 8, 8, 64, 8))
    for tile in [(16, 1, 1, 4), (16, 4, 4, 4), (16, 2, 4, 4), (32, 1, 1, 4), (32, 2, 2, 4),
                 (32, 4, 1, 4), (32, 2, 1, 8), (32, 1, 2, 8)]:
        assert call_conv_tiled(q, L, *args, tile) == 8, tile      # valid: no GPU here
    for tile in [(8, 1, 1, 4), (16, 3, 1, 4), (16, 1, 8, 4), (16, 1, 1, 8), (32, 1, 4, 4),
                 (32, 4, 2, 4), (32, 4, 1, 8), (32, 1, 1, 2)]:
        assert call_conv_tiled(q, L, *args, tile) == 4, tile      # shapes that are not built
    # 128-channel wave tiles of the 32x32 kernel exist at 8 bits only
    assert call_conv_tiled(q, L, (1, 8, 8, 64), 4, 64, g, (0, None, FAKE, FAKE, None, 0, 15),
                           (1, 8, 8, 64, 4), (32, 4, 1, 4)) == 4
    # eight-wave tiles need 16-byte filter taps (C = 4 bytes at 8 bits is a row walk)
    assert call_conv_tiled(q, L, (1, 8, 8, 4), 8, 32, g, REQ8, (1, 8, 8, 32, 8), (32, 1, 1, 8)) == 4
    assert call_conv_tiled(q, L, (1, 8, 8, 256), 1, 32, g, (1, None, None, None, FAKE, 0, 0),
                           (1, 8, 8, 32, 1), (32, 1, 1, 4)) == 4  # no tiles at one bit
    T, G, E = q.qnn.Tensor, q.qnn.ConvGeom, q.qnn.Epi
    assert L.qnn_conv2d_tiled(ctypes.byref(T(1, 8, 8, 32, 8)), FAKE, 64, FAKE, ctypes.byref(G(*g)),
                              ctypes.byref(E(*REQ8)), None, ctypes.byref(T(1, 8, 8, 64, 8)), FAKE,
                              None) == 1


def test_unsupported_local_memory(q, L):
    """A filter bank too long for one local-memory tile is refused on the host."""
    st = call_conv(q, L, (1, 8, 8, 4096), 8, 16, (3, 3, 1, 1, 1, 1), REQ8, (1, 8, 8, 16, 8))
    assert st == 7


def test_batch_zero_is_ok_without_pointers(q, L):
    assert call_conv(q, L, (0, 4, 4, 32), 8, 32, (3, 3, 1, 1, 1, 1), REQ8, (0, 4, 4, 32, 8),
                     xp=None, wp=None, yp=None) == 0


def test_valid_call_without_gpu_reports_device(q, L):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    assert call_conv(q, L, (1, 4, 4, 32), 8, 32, (3, 3, 1, 1, 1, 1), REQ8, (1, 4, 4, 32, 8)) == 8
    assert L.qnn_device_check() == 8


def test_pool_and_relu_validation(q, L):
    T = q.qnn.Tensor
    x = T(1, 4, 4, 32, 8)
    assert L.qnn_maxpool2d(ctypes.byref(T(1, 4, 4, 32, 1)), FAKE, 2, 2, 2, 2,
                           ctypes.byref(T(1, 2, 2, 32, 1)), FAKE, None) == 2
    assert L.qnn_maxpool2d(ctypes.byref(x), FAKE, 0, 2, 2, 2, ctypes.byref(T(1, 2, 2, 32, 8)),
                           FAKE, None) == 4
    assert L.qnn_maxpool2d(ctypes.byref(x), FAKE, 2, 2, 2, 2, ctypes.byref(T(1, 3, 2, 32, 8)),
                           FAKE, None) == 3
    assert L.qnn_maxpool2d(ctypes.byref(x), FAKE, 5, 5, 1, 1, ctypes.byref(T(1, 0, 0, 32, 8)),
                           FAKE, None) == 3
    assert L.qnn_relu_s8(FAKE, FAKE, 0, None) == 0
    assert L.qnn_relu_s8(None, FAKE, 4, None) == 1
    assert L.qnn_relu_s8(FAKE + 1, FAKE, 4, None) == 5


def test_linear_validation(q, L):
    T, E = q.qnn.Tensor, q.qnn.Epi
    x = T(4, 4, 4, 64, 8)
    e = E(2, None, None, None, None, 0, 0)
    assert L.qnn_linear(ctypes.byref(x), FAKE, 10, FAKE, ctypes.byref(e),
                        ctypes.byref(T(4, 1, 2, 10, 32)), FAKE, None) == 3
    assert L.qnn_linear(ctypes.byref(x), FAKE, 10, FAKE, ctypes.byref(e),
                        ctypes.byref(T(4, 1, 1, 10, 8)), FAKE, None) == 2


@pytest.mark.parametrize("bits", [1, 2, 4, 8])
def test_host_pack_unpack_agree_with_generator_and_oracle(q, orc, bits):
    rng = np.random.default_rng(bits)
    for count in (1, 5, 8, 33, 1000):
        codes = rng.integers(0, 1 << bits, size=count)
        packed = q.pack_host(codes.astype(np.uint8), bits)
        assert np.array_equal(packed, synth.pack_codes(codes[None, :], bits)[0])
        for signed in (False, True):
            assert np.array_equal(q.unpack_host(packed, count, bits, signed),
                                  orc.unpack(packed, count, bits, signed))


def test_host_pack_rejects_out_of_range(q, L):
    codes = np.array([0, 16], dtype=np.uint8)
    out = np.zeros(1, dtype=np.uint8)
    assert L.qnn_pack_host(codes.ctypes.data_as(ctypes.c_void_p), 2, 4,
                           out.ctypes.data_as(ctypes.c_void_p)) == 4
    assert L.qnn_pack_host(codes.ctypes.data_as(ctypes.c_void_p), 2, 3,
                           out.ctypes.data_as(ctypes.c_void_p)) == 2


def test_conv_fp4_validation(q, L):
    """The e2m1 (FP4) path: INT-2 only, built tile shapes or (0, 0, 0) for the
    library's pick, filter volume bounded by the exact fp32 range."""
    g = (3, 3, 1, 1, 1, 1)
    REQ2 = (0, None, FAKE, FAKE, None, 0, 3)
    args = ((1, 8, 8, 64), 2, 64, g, REQ2, (1, 8, 8, 64, 2))
    fp4 = q.TILE_FP4
    for tile in [(fp4, 0, 0, 0), (fp4, 1, 1, 4), (fp4, 2, 2, 4), (fp4, 2, 1, 8), (fp4, 2, 2, 8)]:
        assert call_conv_tiled(q, L, *args, tile) == 8, tile      # valid: no GPU here
    for tile in [(fp4, 4, 1, 4), (fp4, 1, 4, 4), (fp4, 0, 1, 0), (fp4, 1, 1, 2), (fp4, 1, 1, 0)]:
        assert call_conv_tiled(q, L, *args, tile) == 4, tile      # shapes that are not built
    # 1-bit layers: the e2m1 path only (binary threshold or raw sums)
    TH1 = (1, None, None, None, FAKE, 0, 0)
    assert call_conv_tiled(q, L, (1, 8, 8, 64), 1, 64, g, TH1, (1, 8, 8, 64, 1), (fp4, 0, 0, 0)) == 8
    assert call_conv_tiled(q, L, (1, 8, 8, 64), 1, 64, g, TH1, (1, 8, 8, 64, 1), (fp4, 1, 2, 8)) == 8
    assert call_conv_tiled(q, L, (1, 8, 8, 64), 1, 64, g, TH1, (1, 8, 8, 64, 1), (32, 1, 1, 4)) == 4
    # 8- and 4-bit layers have no e2m1 form
    assert call_conv_tiled(q, L, (1, 8, 8, 32), 8, 64, g, REQ8, (1, 8, 8, 64, 8), (fp4, 0, 0, 0)) == 2
    assert call_conv_tiled(q, L, (1, 8, 8, 64), 4, 64, g, (0, None, FAKE, FAKE, None, 0, 15),
                           (1, 8, 8, 64, 4), (fp4, 1, 1, 4)) == 2
    # eight waves need whole 16-byte chunks of e2m1 pixels: 32 channels
    assert call_conv_tiled(q, L, (1, 8, 8, 16), 2, 64, g, REQ2, (1, 8, 8, 64, 2), (fp4, 1, 1, 8)) == 4
    # 9 * 310720 = 2796480 > 2^24 / 6: partial sums could leave the exact fp32 range
    big = ((1, 3, 3, 310720), 2, 32, g, REQ2, (1, 3, 3, 32, 2))
    assert call_conv_tiled(q, L, *big, (fp4, 0, 0, 0)) == 6


def test_conv_image_validation(q, L):
    """The whole-image kernel (QNN_TILE_IMAGE): only the (0, 0, 0) shape,
    only for layers it covers (refused on the host otherwise)."""
    img = q.TILE_IMAGE
    REQ2 = (0, None, FAKE, FAKE, None, 0, 3)
    REQ4 = (0, None, FAKE, FAKE, None, 0, 15)
    g5 = (5, 5, 1, 1, 2, 2)
    g3 = (3, 3, 1, 1, 1, 1)
    ok8 = ((2, 32, 32, 4), 8, 32, g5, REQ8, (2, 32, 32, 32, 8))
    assert call_conv_tiled(q, L, *ok8, (img, 0, 0, 0)) == 8               # valid: no GPU here
    for args in [((2, 16, 16, 16), 2, 32, g3, REQ2, (2, 16, 16, 32, 2)),   # one-word pixels
                 ((2, 16, 16, 32), 8, 32, g5, REQ8, (2, 16, 16, 32, 8)),   # 32-byte pixels, 5x5
                 ((2, 8, 8, 32), 4, 64, g5, REQ4, (2, 8, 8, 64, 4)),       # 16-byte pixels, 8-wide
                 ((1, 8, 30, 64), 4, 32, g3, REQ4, (1, 8, 30, 32, 4)),     # 32-byte pixels, 3x3
                 ((1, 9, 16, 64), 2, 32, g3, REQ2, (1, 9, 16, 32, 2)),     # 16-byte pixels at 2 bits
                 ((1, 17, 17, 32), 8, 32, g3, REQ8, (1, 17, 17, 32, 8)),   # 9248-byte image: row bands
                 ((2, 32, 32, 64), 4, 64, g3, REQ4, (2, 32, 32, 64, 4))]:  # row bands, 2 channel groups
        assert call_conv_tiled(q, L, *args, (img, 0, 0, 0)) == 8, args
    for tile in [(img, 1, 0, 0), (img, 0, 1, 0), (img, 0, 0, 4)]:
        assert call_conv_tiled(q, L, *ok8, tile) == 4, tile               # not built
    refused = [
        ((1, 9, 9, 4), 8, 32, (3, 3, 2, 2, 1, 1), REQ8, (1, 5, 5, 32, 8)),     # stride 2
        ((1, 9, 9, 8), 8, 32, g3, REQ8, (1, 9, 9, 32, 8)),                     # 8-byte pixels
        ((1, 9, 9, 16), 8, 32, g3, REQ8, (1, 9, 9, 32, 8)),                    # 16-byte pixels at 8 bits
        ((1, 9, 40, 4), 8, 32, g3, REQ8, (1, 9, 40, 32, 8)),                   # 40 outputs per row
        ((1, 9, 9, 4), 8, 32, (7, 7, 1, 1, 3, 3), REQ8, (1, 9, 9, 32, 8)),     # 7x7 filter
        ((1, 9, 9, 16), 2, 24, g3, REQ2, (1, 9, 9, 24, 2)),                    # 48-bit output pixels
        ((1, 65, 32, 4), 8, 32, g3, REQ8, (1, 65, 32, 32, 8)),                 # 8320-byte image
        ((1, 9, 9, 64), 8, 32, g5, REQ8, (1, 9, 9, 32, 8)),                    # 5x5 of 64-byte pixels
        ((1, 9, 9, 128), 2, 32, g3, REQ2, (1, 9, 9, 32, 2)),                   # 36 K steps
        ((1, 40, 16, 32), 8, 32, g3, REQ8, (1, 40, 16, 32, 8)),                # 20 KB image, 16-wide rows
        ((1, 40, 20, 64), 4, 32, g5, REQ4, (1, 40, 20, 32, 4)),                # 5x5 bands of 2-chunk taps
    ]
    for args in refused:
        assert call_conv_tiled(q, L, *args, (img, 0, 0, 0)) == 7, args
    assert call_conv_tiled(q, L, (1, 8, 8, 32), 1, 32, g3,
                           (1, None, None, None, FAKE, 0, 0), (1, 8, 8, 32, 1), (img, 0, 0, 0)) == 4
