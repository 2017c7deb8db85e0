"""GPU parity of the convolution fused with 2x2 / stride-2 max-pooling
(qnn_conv2d_maxpool) against the oracle's convolution followed by the
oracle's max-pooling, byte for byte."""
import numpy as np
import pytest

import synth
from gpu_helpers import EPI, compare, dev, log, threads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def qnn():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1908_11263_amd as q
    q.device_check()
    return q


def gpu_pool(qnn, L):
    import torch
    y = qnn.conv2d_maxpool(dev(L.x), (L.n, L.h, L.w, L.c), L.bits, dev(L.wt), L.m, L.kh, L.kw,
                           L.stride, L.pad, L.epi, bias=dev(L.bias), mult=dev(L.mult),
                           shift=dev(L.shift), thresh=dev(L.thresh), clip=L.clip)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def oracle_pool(orc, L):
    n = L.n
    _, y = orc.conv2d(L.x, (n, L.h, L.w, L.c), L.bits, L.wt, L.m, L.kh, L.kw, L.stride, L.pad,
                      EPI[L.epi], L.bias, L.mult, L.shift, L.thresh, L.clip, nthreads=threads())
    return orc.maxpool2d(y, (n, L.ho, L.wo, L.m), L.bits, 2, 2, 2, 2)


def check(qnn, orc, L):
    log("case", L.name, L.epi, "pool N=%d H=%d W=%d C=%d M=%d k=%d s=%s p=%s bits=%d" % (
        L.n, L.h, L.w, L.c, L.m, L.kh, L.stride, L.pad, L.bits))
    got = gpu_pool(qnn, L)
    compare(got, oracle_pool(orc, L), "%s %s pool" % (L.name, L.epi))
    return got


def layer(bits, n, h, w, c, m, k, pad=None, stride=1, seed=3, epi="requant"):
    hi = (1 << bits) - 1
    whi = (1 << (bits - 1)) - 1
    pad = k // 2 if pad is None else pad
    span = max(1, k * k * c * hi * whi // 4)
    return synth.conv_layer("pool_int%d" % bits, bits, n, h, w, c, m, k, pad, seed, (0, hi),
                            (-(1 << (bits - 1)), whi), bias_rng=(-hi * 50, hi * 50),
                            mult_rng=(1, 1 << 10), shift=10, clip=(0, hi), epi=epi,
                            stride=stride, thresh_rng=(-span, span))


@pytest.mark.parametrize("bits", [8, 4, 2])
def test_pool_random_small_layers(qnn, orc, bits):
    rng = np.random.default_rng(3000 + bits)
    done = 0
    while done < 14:
        L = synth.random_small_layer(rng, bits, epi="requant")
        if L.ho < 2 or L.wo < 2:
            continue
        check(qnn, orc, L)
        done += 1


@pytest.mark.parametrize("bits", [8, 4, 2])
def test_pool_shapes(qnn, orc, bits):
    unit = 32 // bits
    for (n, h, w, c, m, k, s) in [
            (2, 8, 8, unit, 8, 3, 1),          # narrow layer (fewer than 32 channels)
            (1, 7, 9, unit, 33, 3, 1),         # odd output sizes: last row/column dropped
            (3, 16, 16, 2 * unit, 40, 3, 1),   # whole small images per tile
            (2, 32, 32, unit, 32, 5, 1),       # CIFAR first-layer geometry
            (1, 9, 150, unit, 16, 3, 1),       # rows wider than a tile: 64-column tiles
            (1, 41, 37, unit, 70, 3, 1),       # ragged tiles, odd rows, 3 channel tiles
            (2, 20, 22, 2 * unit, 24, 3, 2),   # strided convolution
            (4, 5, 5, unit, 48, 1, 1)]:        # 1x1 filter, odd image
        check(qnn, orc, layer(bits, n, h, w, c, m, k, stride=s, seed=n * h + m))


@pytest.mark.parametrize("bits", [4, 2])
def test_pool_staircase(qnn, orc, bits):
    unit = 32 // bits
    for (n, h, w, m) in [(2, 9, 8, 12), (24, 32, 32, 64)]:
        L = layer(bits, n, h, w, 2 * unit, m, 3, seed=m, epi="stair")
        check(qnn, orc, L)


@pytest.mark.parametrize("bits", [8, 4])
def test_pool_cifar_layers_batch4096(qnn, orc, bits):
    """The three conv + pool layers of the CIFAR-shaped network at batch 4096
    (whole outputs), fused, against the oracle; the later layers on random
    codes over the whole code range."""
    net = synth.cifar_network(bits=bits, n=4096)
    hw = 32
    rng = np.random.default_rng(17)
    for i, cv in enumerate(net.convs):
        if i == 0:
            x_vals = net.x_vals
        else:
            x_vals = rng.integers(0, net.clip[1] + 1, size=(net.n, hw, hw, cv["c"]))
        L = synth.ConvLayer("cifar%d_conv%d" % (bits, i + 1), bits, net.n, hw, hw, cv["c"], cv["m"],
                            5, 5, (1, 1), (2, 2), "requant", x_vals, cv["w_vals"], cv["bias"],
                            cv["mult"], cv["shift"], None, net.clip, cv["c_alg"])
        check(qnn, orc, L)
        hw //= 2
