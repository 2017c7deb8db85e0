"""GPU parity of the INT-2 and INT-1 paths on the FP4 (e2m1) matrix
instruction (qnn_conv2d_tiled with QNN_TILE_FP4) against the CPU oracle,
byte for byte: random small layers of every geometry class and epilogue,
every FP4 tile shape, accumulators at the extremes of the code ranges, and
the whole outputs of the batch-256 16x16x128 INT-2 layer and the batch-1024
8x8x256 INT-1 layer."""
import numpy as np
import pytest

import synth
from gpu_helpers import compare, dev, log, oracle_conv, with_epi

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def qnn():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1908_11263_amd as q
    q.device_check()
    return q


def fp4_tiles(q):
    return [(q.TILE_FP4, 0, 0, 0)] + [(q.TILE_FP4, m, n, w) for m in (1, 2) for n in (1, 2)
                                      for w in (4, 8)]


def run_fp4(qnn, L, tile=None, epi=None):
    import torch
    epi = epi or L.epi
    tile = tile or (qnn.TILE_FP4, 0, 0, 0)
    y = qnn.conv2d(dev(L.x), (L.n, L.h, L.w, L.c), L.bits, dev(L.wt), L.m, L.kh, L.kw, L.stride,
                   L.pad, epi, bias=dev(L.bias), mult=dev(L.mult), shift=dev(L.shift),
                   thresh=dev(L.thresh), clip=L.clip, tile=tile)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def check(qnn, orc, L, tile=None, epi=None):
    epi = epi or L.epi
    log("case fp4", L.name, epi, "tile", tile, "N=%d H=%d W=%d C=%d M=%d k=%dx%d s=%s p=%s" % (
        L.n, L.h, L.w, L.c, L.m, L.kh, L.kw, L.stride, L.pad))
    got = run_fp4(qnn, L, tile, epi)
    compare(got, oracle_conv(orc, L, epi), "%s %s tile %s" % (L.name, epi, tile))
    return got


@pytest.mark.parametrize("epi", ["requant", "raw32", "stair"])
def test_fp4_random_layers(qnn, orc, epi):
    """16, 32 and 48 channels (row walk, tap walk), strides 1-2, pads 0-2,
    kernels 1-5, 1-40 filters."""
    rng = np.random.default_rng({"requant": 41, "raw32": 42, "stair": 43}[epi])
    for _ in range(16):
        check(qnn, orc, synth.random_small_layer(rng, 2, epi=epi))


def layer(n, h, w, c, m, k, seed, epi="requant"):
    return synth.conv_layer("fp4_int2", 2, n, h, w, c, m, k, k // 2, seed, (0, 3), (-2, 1),
                            bias_rng=(-150, 150), mult_rng=(1, 1 << 10), shift=10, clip=(0, 3),
                            epi=epi, thresh_rng=(-k * k * c // 2, k * k * c // 2))


def test_fp4_every_tile_shape(qnn, orc):
    for L in (layer(3, 13, 17, 64, 70, 3, seed=7), layer(2, 9, 6, 16, 33, 1, seed=8),
              layer(2, 11, 10, 32, 40, 3, seed=9, epi="stair")):
        want = oracle_conv(orc, L)
        for tile in fp4_tiles(qnn):
            log("case fp4", L.name, L.epi, "tile", tile, "C=%d M=%d" % (L.c, L.m))
            if tile[3] == 8 and (L.c % 32 or L.epi == "stair"):
                # eight waves: whole 16-byte e2m1 chunks per tap, plain epilogues
                with pytest.raises(qnn.QnnError) as e:
                    run_fp4(qnn, L, tile)
                assert e.value.status == 4
                continue
            got = run_fp4(qnn, L, tile)
            bad = np.argwhere(got != want)
            assert bad.size == 0, "tile %s: %d mismatches, first at %s" % (tile, len(bad), bad[:5].tolist())


def test_fp4_extreme_accumulators(qnn, orc):
    """Every product at its largest magnitude (x = 3 with w = -2, and with
    w = 1) over the deepest filter that fits: raw sums checked exactly."""
    for wv in (-2, 1):
        L = layer(2, 6, 7, 512, 64, 3, seed=11, epi="raw32")
        x_vals = np.full_like(L.x_vals, 3)
        w_vals = np.full_like(L.w_vals, wv)
        E = synth.ConvLayer("fp4_extreme_w%d" % wv, 2, L.n, L.h, L.w, L.c, L.m, L.kh, L.kw,
                            L.stride, L.pad, "raw32", x_vals, w_vals, L.bias, None, None, None,
                            (0, 0))
        got = check(qnn, orc, E)
        # interior pixels see all 9 taps: 9 * 512 * 3 * w + bias
        inner = got[:, 1:-1, 1:-1, :]
        assert np.array_equal(inner, np.broadcast_to(9 * 512 * 3 * wv + L.bias, inner.shape))


def test_fp4_int2_layer_batch256(qnn, orc):
    """The whole batch-256 INT-2 output on the FP4 path against the oracle:
    the workload's scale-and-clamp, raw sums and the centred variant."""
    L = synth.int2_layer()
    check(qnn, orc, L)
    check(qnn, orc, with_epi(L, "raw32"))
    check(qnn, orc, synth.centred(L))


# ------------------------------------------------------------------ INT-1

@pytest.mark.parametrize("epi", ["thresh1", "raw32"])
def test_fp4_int1_random_layers(qnn, orc, epi):
    """32, 64 and 96 channels, strides 1-2, pads 0-2 (padding taps are -1),
    kernels 1-5, 1-79 filters."""
    rng = np.random.default_rng({"thresh1": 51, "raw32": 52}[epi])
    for _ in range(16):
        check(qnn, orc, synth.random_small_layer(rng, 1, epi=epi))


def int1_layer(n, h, w, c, m, k, seed, epi="thresh1"):
    return synth.conv_layer("fp4_int1", 1, n, h, w, c, m, k, k // 2, seed, None, None,
                            bias_rng=(-20, 20), thresh_rng=(-k * k * c // 4, k * k * c // 4), epi=epi)


def test_fp4_int1_every_tile_shape(qnn, orc):
    for L in (int1_layer(3, 13, 17, 64, 70, 3, seed=21), int1_layer(2, 9, 6, 32, 33, 1, seed=22),
              int1_layer(2, 11, 10, 96, 40, 3, seed=23, epi="raw32")):
        want = oracle_conv(orc, L)
        for tile in fp4_tiles(qnn):
            log("case fp4", L.name, L.epi, "tile", tile, "C=%d M=%d" % (L.c, L.m))
            got = run_fp4(qnn, L, tile)
            bad = np.argwhere(got != want)
            assert bad.size == 0, "tile %s: %d mismatches, first at %s" % (tile, len(bad), bad[:5].tolist())


def test_fp4_int1_extreme_accumulators(qnn, orc):
    """All +1 against all -1 and all +1 over a deep filter: raw sums of
    -K and +K, with the -1 padding taps at the borders."""
    for wv in (-1, 1):
        L = int1_layer(2, 6, 7, 512, 64, 3, seed=24, epi="raw32")
        E = synth.ConvLayer("fp4_int1_extreme_w%d" % wv, 1, L.n, L.h, L.w, L.c, L.m, L.kh, L.kw,
                            L.stride, L.pad, "raw32", np.ones_like(L.x_vals),
                            np.full_like(L.w_vals, wv), L.bias, None, None, None, (0, 0))
        got = check(qnn, orc, E)
        inner = got[:, 1:-1, 1:-1, :]
        assert np.array_equal(inner, np.broadcast_to(9 * 512 * wv + L.bias, inner.shape))


def test_fp4_int1_layer_batch1024(qnn, orc):
    """The whole batch-1024 INT-1 output on the FP4 path against the oracle:
    binary thresholds and raw sums."""
    L = synth.int1_layer()
    check(qnn, orc, L)
    check(qnn, orc, with_epi(L, "raw32"))


def test_fp4_workgroups_walk_several_tiles(qnn, orc):
    """The library's FP4 plan (eight-wave tiles, one workgroup per compute
    unit walking its channel group's tiles) with more tiles than workgroups,
    an uneven split and a ragged last tile: 301 images of 8x8x256 at 1 bit
    (76 tiles of four images for 64 workgroups per channel group), and 520
    images of 16x16x128 at 2 bits with 64 filters (260 tiles of two images
    for 256 workgroups)."""
    check(qnn, orc, int1_layer(301, 8, 8, 256, 256, 3, seed=25))
    check(qnn, orc, layer(520, 16, 16, 128, 64, 3, seed=26))
