"""GPU parity of the whole-image convolution kernel (QNN_TILE_IMAGE: small
images whose padded tiles fit in local memory -- a network's first layer
with one-word pixels, and layers of 8- to 32-pixel-wide images with 16- or
32-byte pixels) against the CPU oracle, byte for byte: plain and pooled
scale-and-clamp, raw accumulators, every compression-plan mode (including
multipliers that are not positive, where pooling must follow the
compression), odd and ragged image sizes, images loaded word by word,
several images per workgroup step, many steps per workgroup, and layers
the kernel must refuse."""
import numpy as np
import pytest

import synth
from gpu_helpers import EPI, dev, log, oracle_conv, threads

pytestmark = pytest.mark.gpu

IMAGE = (1, 0, 0, 0)


@pytest.fixture(scope="module")
def qnn():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1908_11263_amd as q
    q.device_check()
    return q


def layer(bits, n, h, w, m, k, pad, seed, epi="requant", mult_rng=(1, 1 << 10), shift=10,
          clip=None, c=None):
    """One-word pixels (32/bits channels) unless c is given."""
    hi = (1 << bits) - 1
    whi = (1 << (bits - 1)) - 1
    c = c or 32 // bits
    return synth.conv_layer("img_int%d_c%d" % (bits, c), bits, n, h, w, c, m, k, pad, seed, (0, hi),
                            (-(1 << (bits - 1)), whi), bias_rng=(-hi * 50, hi * 50),
                            mult_rng=mult_rng, shift=shift, clip=clip or (0, hi), epi=epi)


def run(qnn, L, pool=False, tile=None, epi=None):
    import torch
    epi = epi or L.epi
    args = (dev(L.x), (L.n, L.h, L.w, L.c), L.bits, dev(L.wt), L.m, L.kh, L.kw, L.stride, L.pad, epi)
    kw = dict(bias=dev(L.bias), mult=dev(L.mult), shift=dev(L.shift), clip=L.clip)
    if L.thresh is not None:
        kw["thresh"] = dev(L.thresh)
    if pool:
        assert tile is None
        y = qnn.conv2d_maxpool(*args, **kw)
    else:
        y = qnn.conv2d(*args, tile=tile, **kw)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def want(orc, L, pool=False, epi=None):
    y = oracle_conv(orc, L, epi=epi)
    if pool:
        y = orc.maxpool2d(y, (L.n, L.ho, L.wo, L.m), L.bits, 2, 2, 2, 2)
    return y


def check(qnn, orc, L, pool=False, epi=None, tile=None):
    log("case", L.name, epi or L.epi, "pool" if pool else "", "tile", tile,
        "N=%d H=%d W=%d M=%d k=%d p=%s" % (L.n, L.h, L.w, L.m, L.kh, L.pad))
    got = run(qnn, L, pool=pool, tile=tile, epi=epi)
    ref = want(orc, L, pool=pool, epi=epi)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    bad = np.argwhere(got != ref)
    assert bad.size == 0, "%s: %d mismatches, first at %s" % (L.name, len(bad), bad[:5].tolist())


# (n, h, w, m, k, pad): CIFAR-like first layers, narrow outputs, odd and
# ragged sizes (h*w not a multiple of 4: word-by-word image loads), wide
# padding, several channel groups
SHAPES = [
    (3, 32, 32, 32, 5, 2),
    (5, 28, 28, 64, 5, 0),
    (2, 17, 13, 96, 3, 1),
    (7, 8, 8, 32, 3, 3),
    (1, 30, 32, 48, 5, 2),
    (4, 9, 31, 16, 3, 0),
    (2, 1, 1, 32, 3, 1),
]


@pytest.mark.parametrize("bits", [8, 4, 2])
@pytest.mark.parametrize("pool", [False, True])
def test_img_requant(qnn, orc, bits, pool):
    for i, (n, h, w, m, k, pad) in enumerate(SHAPES):
        if m * bits % 32:
            continue
        L = layer(bits, n, h, w, m, k, pad, seed=100 * bits + i)
        if pool and (L.ho < 2 or L.wo < 2):
            continue
        check(qnn, orc, L, pool=pool)
        if not pool:
            # the library's choice is this kernel: forcing it gives the same bytes
            check(qnn, orc, L, tile=IMAGE)


@pytest.mark.parametrize("pool", [False, True])
def test_img_half_word_pixels(qnn, orc, pool):
    """2-byte pixels (4 channels at 4 bits: a network's first layer with 3
    image channels and a zero channel): requantized, pooled, raw sums and the
    staircase, over the first-layer shapes (ragged sizes load the image
    half-word by half-word)."""
    for i, (n, h, w, m, k, pad) in enumerate(SHAPES):
        L = layer(4, n, h, w, m, k, pad, seed=300 + i, c=4)
        if pool and (L.ho < 2 or L.wo < 2):
            continue
        check(qnn, orc, L, pool=pool)
        if not pool:
            check(qnn, orc, L, epi="raw32")
            check(qnn, orc, L, tile=IMAGE)
    for i, (n, h, w, m, k, pad) in enumerate(SHAPES[:4]):
        S = stair_img_layer(4, 4, n, h, w, m, k, pad, seed=310 + i, sorted_=i % 2 == 0)
        if pool and (S.ho < 2 or S.wo < 2):
            continue
        check(qnn, orc, S, pool=pool)


@pytest.mark.parametrize("bits", [8, 4, 2])
def test_img_raw32(qnn, orc, bits):
    for i, (n, h, w, m, k, pad) in enumerate(SHAPES):
        if m * bits % 32:
            continue
        check(qnn, orc, layer(bits, n, h, w, m, k, pad, seed=7 + i), epi="raw32")


@pytest.mark.parametrize("bits", [8, 4, 2])
def test_img_plan_modes(qnn, orc, bits):
    """Multipliers above 2^shift (the general plan forms), shift 0 and clip
    bounds inside the code range, multipliers that are zero or negative
    (the compression is not monotone: codes are pooled after it), and the
    largest shift the plans take (30) with small and large multipliers, whose
    threshold quotients reach 2^38 (the plans' floor divisions at the top of
    their range)."""
    hi = (1 << bits) - 1
    cases = [dict(mult_rng=(1 << 12, 1 << 14), shift=8),
             dict(mult_rng=(1, 3), shift=0, clip=(1, hi - 1) if hi > 2 else (0, hi)),
             dict(mult_rng=(-(1 << 10), 1 << 10), shift=9),
             dict(mult_rng=((1 << 30), (1 << 31) - 1), shift=40),
             dict(mult_rng=(1, 1 << 8), shift=30),
             dict(mult_rng=((1 << 29), (1 << 30)), shift=30),
             dict(mult_rng=(1 << 20, 1 << 22), shift=24)]
    for j, kw in enumerate(cases):
        L = layer(bits, 3, 12, 14, 32, 3, 1, seed=50 + j, **kw)
        check(qnn, orc, L)
        check(qnn, orc, L, pool=True)


@pytest.mark.parametrize("bits", [8, 4])
def test_img_many_images(qnn, orc, bits):
    """More images than workgroups: every workgroup walks several images
    with the next image's words prefetched."""
    L = layer(bits, 2500, 16, 16, 32, 3, 1, seed=bits)
    check(qnn, orc, L, pool=True)


def test_img_equals_general_kernels(qnn, orc):
    """The same layer through the one-word-pixel kernel and through the
    general 32x32 and 16x16 tiles."""
    for bits in (8, 4, 2):
        L = layer(bits, 2, 32, 32, 32, 5, 2, seed=bits)
        ref = want(orc, L)
        for tile in (IMAGE, (32, 1, 2, 4), (16, 2, 1, 4)):
            assert np.array_equal(run(qnn, L, tile=tile), ref), (bits, tile)


def test_img_refuses_layers_it_does_not_cover(qnn, orc):
    """Forced on a layer outside its domain the kernel is refused with
    QNN_ERR_UNSUPPORTED (7); the library's own choice still matches."""
    L8 = layer(8, 1, 9, 9, 32, 3, 1, seed=1)
    outside = [
        synth.conv_layer("img_stride2", 8, 1, 9, 9, 4, 32, 3, 1, 2, (0, 255), (-128, 127),
                         bias_rng=(-99, 99), mult_rng=(1, 1 << 10), shift=10, clip=(0, 255),
                         stride=2),                                        # stride 2
        synth.conv_layer("img_c8", 8, 1, 9, 9, 8, 32, 3, 1, 2, (0, 255), (-128, 127),
                         bias_rng=(-99, 99), mult_rng=(1, 1 << 10), shift=10, clip=(0, 255)),  # 8-byte pixels
        layer(8, 1, 9, 9, 32, 5, 2, seed=5, c=64),                         # 5x5, 64-byte pixels
        layer(4, 1, 9, 9, 32, 5, 2, seed=6, c=64),                         # 5x5, 2 chunks per tap
        layer(2, 1, 9, 9, 32, 3, 1, seed=7, c=128),                        # 3x3, 4 chunks per tap
        layer(8, 1, 9, 40, 32, 3, 1, seed=2),                              # rows of 40 outputs
        layer(8, 1, 9, 9, 32, 1, 0, seed=3),                               # 1x1 filter
        layer(2, 1, 9, 9, 24, 3, 1, seed=4),                               # 24 channels at 2 bits
    ]
    for L in outside:
        with pytest.raises(qnn.QnnError) as e:
            run(qnn, L, tile=IMAGE)
        assert e.value.status == 7, L.name
        check(qnn, orc, L)
    with pytest.raises(qnn.QnnError) as e:
        run(qnn, with_stair(L8), tile=IMAGE)
    assert e.value.status in (2, 7)


def with_stair(L):
    return synth.ConvLayer(L.name + "_stair", L.bits, L.n, L.h, L.w, L.c, L.m, L.kh, L.kw,
                           L.stride, L.pad, "stair", L.x_vals, L.w_vals, L.bias, None, None,
                           np.zeros((L.m, (1 << L.bits) - 1), np.int32), L.clip, L.c_alg)


# (bits, channels, n, h, w, m, k, pad): 16- and 32-byte pixels, output rows
# of 8, 16 and up to 32 pixels, ragged sizes, several 32-channel groups, and
# the CIFAR-shaped network's second and third layers
WIDE = [
    (8, 32, 3, 16, 16, 32, 5, 2),
    (8, 32, 5, 8, 8, 64, 5, 2),
    (8, 32, 2, 13, 11, 40, 3, 1),
    (8, 32, 2, 7, 30, 32, 3, 1),
    (8, 32, 1, 16, 16, 32, 3, 1),
    (4, 32, 3, 16, 16, 32, 5, 2),
    (4, 32, 6, 8, 8, 64, 5, 2),
    (4, 64, 2, 12, 9, 24, 3, 1),
    (4, 64, 2, 5, 26, 64, 3, 1),
    (4, 32, 2, 21, 17, 48, 3, 0),
    (2, 64, 3, 9, 16, 32, 3, 1),
    (2, 64, 2, 6, 6, 48, 3, 2),
]


@pytest.mark.parametrize("pool", [False, True])
def test_img_wide_pixels(qnn, orc, pool):
    for i, (bits, c, n, h, w, m, k, pad) in enumerate(WIDE):
        L = layer(bits, n, h, w, m, k, pad, seed=300 + i, c=c)
        if pool and (L.ho < 2 or L.wo < 2):
            continue
        check(qnn, orc, L, pool=pool)
        if not pool:
            check(qnn, orc, L, tile=IMAGE)
            check(qnn, orc, L, epi="raw32")


@pytest.mark.parametrize("bits", [8, 4])
def test_img_wide_plan_modes(qnn, orc, bits):
    """The general plan forms and non-positive multipliers on 32-channel
    16x16 and 8x8 images."""
    hi = (1 << bits) - 1
    for j, kw in enumerate([dict(mult_rng=(1 << 12, 1 << 14), shift=8),
                            dict(mult_rng=(1, 3), shift=0, clip=(1, hi - 1)),
                            dict(mult_rng=(-(1 << 10), 1 << 10), shift=9)]):
        for (h, w) in ((16, 16), (8, 8)):
            L = layer(bits, 3, h, w, 32, 5, 2, seed=70 + j, c=32, **kw)
            check(qnn, orc, L)
            check(qnn, orc, L, pool=True)


@pytest.mark.parametrize("bits", [8, 4])
def test_img_wide_many_images(qnn, orc, bits):
    """More image groups than workgroups, four 8x8 images per step."""
    L = layer(bits, 3001, 8, 8, 64, 5, 2, seed=bits, c=32)
    check(qnn, orc, L, pool=True)


# (bits, channels, n, h, w, m, k, pad): images larger than one tile, walked
# in bands of 8 output rows: the INT-4 batch-64 layer's shape, 5x5 filters,
# ragged heights (a partial last band), rows of 17 to 32 outputs, no
# padding and padding wider than the filter's half (halo rows above and
# below the image in two bands), several and partial 32-channel groups
BANDS = [
    (4, 64, 2, 32, 32, 64, 3, 1),
    (8, 32, 2, 32, 32, 32, 3, 1),
    (8, 32, 2, 32, 32, 32, 5, 2),
    (8, 32, 3, 27, 19, 40, 5, 2),
    (4, 64, 2, 41, 23, 96, 3, 1),
    (4, 64, 1, 20, 30, 32, 3, 0),
    (8, 32, 1, 18, 17, 32, 3, 1),
    (8, 32, 2, 30, 32, 64, 5, 0),
    (8, 32, 1, 20, 26, 32, 3, 3),
]


@pytest.mark.parametrize("pool", [False, True])
def test_img_bands(qnn, orc, pool):
    for i, (bits, c, n, h, w, m, k, pad) in enumerate(BANDS):
        L = layer(bits, n, h, w, m, k, pad, seed=500 + i, c=c)
        assert L.h * L.w * L.c * bits // 8 > 8192
        check(qnn, orc, L, pool=pool)
        if not pool:
            check(qnn, orc, L, tile=IMAGE)
            check(qnn, orc, L, epi="raw32")


@pytest.mark.parametrize("bits", [8, 4])
def test_img_band_plan_modes(qnn, orc, bits):
    """The general plan forms and non-positive multipliers in band mode."""
    hi = (1 << bits) - 1
    c = 256 // bits
    for j, kw in enumerate([dict(mult_rng=(1 << 12, 1 << 14), shift=8),
                            dict(mult_rng=(1, 3), shift=0, clip=(1, hi - 1)),
                            dict(mult_rng=(-(1 << 10), 1 << 10), shift=9)]):
        L = layer(bits, 2, 26, 24, 32, 3, 1, seed=90 + j, c=c, **kw)
        check(qnn, orc, L)
        check(qnn, orc, L, pool=True)


@pytest.mark.parametrize("bits", [8, 4])
def test_img_band_many_steps(qnn, orc, bits):
    """More bands than resident workgroups: workgroups walk several bands of
    different images, each prefetched during the previous one."""
    L = layer(bits, 300, 18, 17, 32, 3, 1, seed=40 + bits, c=256 // bits)
    check(qnn, orc, L)


def stair_img_layer(bits, c, n, h, w, m, k, pad, seed, sorted_=True):
    """Staircase layer (Sec. III-A, Eq. (4)): 2^bits - 1 thresholds per
    channel over a quarter of the accumulator range, sorted or not."""
    hi = (1 << bits) - 1
    whi = (1 << (bits - 1)) - 1
    span = max(1, k * k * c * hi * whi // 4)
    return synth.conv_layer("img_stair_int%d_c%d" % (bits, c), bits, n, h, w, c, m, k, pad, seed, (0, hi),
                            (-(1 << (bits - 1)), whi), bias_rng=(-hi * 64, hi * 64),
                            thresh_rng=(-span, span), epi="stair", stair_sorted=sorted_)


# (bits, channels, n, h, w, m, k, pad): one-word pixels (a first layer's
# shape; ragged, two channel groups), 16- and 32-byte pixels (5x5, a partial
# group), and row bands (the INT-4 batch-64 layer's shape, a ragged band)
STAIR = [
    (4, 8, 3, 32, 32, 32, 5, 2),
    (2, 16, 2, 17, 13, 64, 3, 1),
    (4, 32, 3, 16, 16, 32, 5, 2),
    (4, 64, 2, 12, 9, 24, 3, 1),
    (2, 64, 3, 9, 16, 32, 3, 1),
    (4, 64, 2, 32, 32, 64, 3, 1),
    (4, 64, 1, 27, 19, 40, 3, 1),
]


@pytest.mark.parametrize("pool", [False, True])
def test_img_stair(qnn, orc, pool):
    """The staircase epilogue on the image kernel, plain and fused with
    pooling (taken on the accumulators: the level is non-decreasing in the
    accumulator for any thresholds), forced and by the library's choice."""
    for i, (bits, c, n, h, w, m, k, pad) in enumerate(STAIR):
        L = stair_img_layer(bits, c, n, h, w, m, k, pad, seed=600 + i)
        if pool and (L.ho < 2 or L.wo < 2):
            continue
        check(qnn, orc, L, pool=pool)
        if not pool:
            check(qnn, orc, L, tile=IMAGE)


def test_img_stair_unsorted(qnn, orc):
    """Unsorted thresholds: the output counts the thresholds at or below the
    biased accumulator."""
    for i, (bits, c, n, h, w, m, k, pad) in enumerate(STAIR[::2]):
        L = stair_img_layer(bits, c, n, h, w, m, k, pad, seed=700 + i, sorted_=False)
        check(qnn, orc, L, tile=IMAGE)
        if L.ho >= 2 and L.wo >= 2:
            check(qnn, orc, L, pool=True)



def test_img_stair_ties_and_extremes(qnn, orc):
    """Sorted thresholds with ties (every odd threshold equal to its left
    neighbour) and thresholds far outside the accumulator range, whose
    scaled form clamps to the int32 limits: a channel whose thresholds all
    lie below every accumulator (code 2^b - 1 throughout), one whose
    thresholds all lie above (code 0), and random runs of extremes at both
    ends of the others.  The comparison tree must count exactly at equal
    thresholds and at the clamped ends."""
    import dataclasses
    lo, hi = -(1 << 31), (1 << 31) - 1
    cases = [(4, 64, 2, 32, 32, 64, 3, 1), (4, 64, 1, 12, 9, 40, 3, 1), (2, 64, 2, 9, 16, 32, 3, 1)]
    for i, (bits, c, n, h, w, m, k, pad) in enumerate(cases):
        L = stair_img_layer(bits, c, n, h, w, m, k, pad, seed=800 + i)
        rng = np.random.default_rng(900 + i)
        t = L.thresh.astype(np.int64)
        t[:, 1::2] = t[:, 0:-1:2]
        nt = t.shape[1]
        for j in range(2, m):
            r, s = rng.integers(0, 3), rng.integers(0, 4)
            t[j, :r] = lo
            if s:
                t[j, nt - s:] = hi
        t[0, :] = lo
        t[1, :] = hi
        t = np.sort(t, axis=1)
        L2 = dataclasses.replace(L, name=L.name + "_ties", thresh=t.astype(np.int32))
        check(qnn, orc, L2, tile=IMAGE)
        check(qnn, orc, L2)
        if L2.ho >= 2 and L2.wo >= 2:
            check(qnn, orc, L2, pool=True)
