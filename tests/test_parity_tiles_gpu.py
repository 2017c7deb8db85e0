"""GPU parity of every built tile shape (qnn_conv2d_tiled) against the CPU
oracle: both int8-MFMA kernels, each wave-tile size, four- and eight-wave
workgroups, on layers with ragged channel counts and image sizes."""
import numpy as np
import pytest

import synth
from gpu_helpers import dev, log, oracle_conv

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def qnn():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1908_11263_amd as q
    q.device_check()
    return q


def tiles(bits):
    out = [(16, m, n, 4) for m in (1, 2, 4) for n in (1, 2, 4)]
    out += [(32, m, n, w) for m in (1, 2) for n in (1, 2) for w in (4, 8)]
    if bits == 8:
        out.append((32, 4, 1, 4))
    return out


def run_tiled(qnn, L, tile, epi=None):
    import torch
    epi = epi or L.epi
    y = qnn.conv2d(dev(L.x), (L.n, L.h, L.w, L.c), L.bits, dev(L.wt), L.m, L.kh, L.kw, L.stride,
                   L.pad, epi, bias=dev(L.bias), mult=dev(L.mult), shift=dev(L.shift),
                   thresh=dev(L.thresh), clip=L.clip, tile=tile)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def layer(bits, n, h, w, cu, m, k, seed, epi="requant"):
    hi = (1 << bits) - 1
    whi = (1 << (bits - 1)) - 1
    c = cu * 32 // bits
    return synth.conv_layer("tiles_int%d" % bits, bits, n, h, w, c, m, k, k // 2, seed, (0, hi),
                            (-(1 << (bits - 1)), whi), bias_rng=(-hi * 50, hi * 50),
                            mult_rng=(1, 1 << 10), shift=10, clip=(0, hi), epi=epi,
                            thresh_rng=(-k * k * c * hi * whi // 4, k * k * c * hi * whi // 4))


@pytest.mark.parametrize("bits", [8, 4, 2])
def test_every_tile_shape(qnn, orc, bits):
    # a multiple of 16 channels (tap walk) and fewer (row walk)
    for L in (layer(bits, 3, 13, 17, 4, 70, 3, seed=bits), layer(bits, 2, 9, 6, 1, 33, 1, seed=5)):
        want = oracle_conv(orc, L)
        for tile in tiles(bits):
            log("case", L.name, "tile", tile, "M=%d H=%d W=%d C=%d" % (L.m, L.h, L.w, L.c))
            if tile[3] == 8 and L.c % 16:
                # eight-wave tiles walk K tap by tap, which needs a multiple
                # of 16 channels (codes are widened to bytes when staged)
                with pytest.raises(qnn.QnnError) as e:
                    run_tiled(qnn, L, tile)
                assert e.value.status == 4
                continue
            got = run_tiled(qnn, L, tile)
            bad = np.argwhere(got != want)
            assert bad.size == 0, "tile %s: %d mismatches, first at %s" % (tile, len(bad), bad[:5].tolist())


@pytest.mark.parametrize("bits", [4, 2])
def test_tile_shapes_raw_and_staircase(qnn, orc, bits):
    for epi in ("raw32", "stair"):
        L = layer(bits, 2, 11, 10, 4, 40, 3, seed=9, epi=epi)
        want = oracle_conv(orc, L)
        for tile in tiles(bits):
            log("case", L.name, epi, "tile", tile)
            if epi == "stair" and tile[3] == 8:
                # eight-wave tiles are built for scale-and-clamp and raw layers
                with pytest.raises(qnn.QnnError) as e:
                    run_tiled(qnn, L, tile)
                assert e.value.status == 4
                continue
            assert np.array_equal(run_tiled(qnn, L, tile), want), tile


def test_tile_shape_not_fitting_is_refused(qnn):
    """A filter tile too long for the local memory: QNN_ERR_UNSUPPORTED, and
    nothing is launched."""
    L = layer(8, 1, 4, 4, 64, 64, 3, seed=1)   # K = 9 * 2048 bytes per filter row
    with pytest.raises(qnn.QnnError) as e:
        run_tiled(qnn, L, (16, 4, 1, 4))
    assert e.value.status == 7
