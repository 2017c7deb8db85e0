"""GPU parity: the HIP path (called through the C ABI) against the CPU oracle
on the same seeded inputs, byte for byte (integer work: no tolerance)."""
import numpy as np
import pytest

import synth
from gpu_helpers import compare, dev, distribution, gpu_conv, log, oracle_conv, threads, with_epi

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def qnn():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1908_11263_amd as q
    q.device_check()
    return q


def check_layer(orc, L, epi=None):
    """The whole output of layer L on the GPU against the oracle's."""
    epi = epi or L.epi
    log("case", L.name, epi, "N=%d H=%d W=%d C=%d M=%d k=%dx%d s=%s p=%s bits=%d" % (
        L.n, L.h, L.w, L.c, L.m, L.kh, L.kw, L.stride, L.pad, L.bits))
    got = gpu_conv(L, epi)
    compare(got, oracle_conv(orc, L, epi), "%s %s" % (L.name, epi))
    return got


# ------------------------------------------------------ the five workloads

def test_int8_layer_batch1(qnn, orc):
    L = synth.int8_layer()
    y = check_layer(orc, L)
    log("int8 distribution (zero, top):", distribution(y, 8))
    check_layer(orc, with_epi(L, "raw32"))


def test_int4_layer_batch64(qnn, orc):
    L = synth.int4_layer()
    check_layer(orc, L)
    check_layer(orc, with_epi(L, "raw32"))
    C = synth.centred(L)
    y = check_layer(orc, C)
    z, top = distribution(y, 4)
    log("int4 centred distribution (zero, top):", z, top)
    assert 0.2 < z < 0.8


def test_int2_layer_batch256(qnn, orc):
    L = synth.int2_layer()
    check_layer(orc, L)
    check_layer(orc, with_epi(L, "raw32"))
    C = synth.centred(L)
    y = check_layer(orc, C)
    z, top = distribution(y, 2)
    log("int2 centred distribution (zero, top):", z, top)
    assert 0.2 < z < 0.8


def test_int1_layer_batch1024(qnn, orc):
    L = synth.int1_layer()
    check_layer(orc, L)
    check_layer(orc, with_epi(L, "raw32"))


def oracle_network(orc, net):
    """The network on the oracle, layer by layer (convolution, then
    max-pooling), over the whole batch: (logits [n, 10], pooled activations
    of each layer)."""
    x = net.packed_input()
    n = x.shape[0]
    h, c = 32, x.shape[-1] * 8 // net.bits
    acts = []
    for cv in net.convs:
        wt = synth.pack_codes(synth.to_code(cv["w_vals"], net.bits, True).reshape(cv["m"], -1),
                              net.bits)
        _, y = orc.conv2d(x, (n, h, h, c), net.bits, wt, cv["m"], 5, 5, (1, 1), (2, 2), 0,
                          cv["bias"], cv["mult"], cv["shift"], None, net.clip, nthreads=threads())
        c = cv["m"]
        x = orc.maxpool2d(y, (n, h, h, c), net.bits, 2, 2, 2, 2)
        acts.append(x)
        h //= 2
    fcw = synth.pack_codes(synth.to_code(net.fc_w_vals, net.bits, True), net.bits)
    _, logits = orc.linear(x, n, h * h * c, net.bits, fcw, 10, epi=2, bias=net.fc_bias)
    return logits, acts


def gpu_network(qnn, net, fused=True):
    """The network on the GPU: (logits [n, 10], the layers' pooled outputs)."""
    import torch
    from paper_1908_11263_amd.network import cifar_forward
    convs = []
    for cv in net.convs:
        wt = synth.pack_codes(synth.to_code(cv["w_vals"], net.bits, True).reshape(cv["m"], -1),
                              net.bits)
        convs.append(dict(w=dev(wt), bias=dev(cv["bias"]), mult=dev(cv["mult"]),
                          shift=dev(cv["shift"]), m=cv["m"], k=5, pad=2))
    fc = dict(w=dev(synth.pack_codes(synth.to_code(net.fc_w_vals, net.bits, True), net.bits)),
              bias=dev(net.fc_bias), m=10)
    x = dev(net.packed_input())
    cin = net.x_vals.shape[-1]
    logits, acts = cifar_forward(x, net.n, net.bits, cin, convs, fc, net.clip, fused=fused,
                                 keep=True)
    torch.cuda.synchronize()
    pooled = acts if fused else acts[1::2]
    return logits.cpu().numpy().reshape(net.n, 10), [a.cpu().numpy() for a in pooled]


def check_network(qnn, orc, net, fused=True):
    log("case cifar network bits=%d N=%d fused=%s" % (net.bits, net.n, fused))
    want, want_acts = oracle_network(orc, net)
    got, got_acts = gpu_network(qnn, net, fused=fused)
    for i, (g, w) in enumerate(zip(got_acts, want_acts)):
        compare(g, w, "cifar%d layer %d (conv + pool)" % (net.bits, i + 1))
    compare(got, want, "cifar%d logits" % net.bits)


@pytest.mark.parametrize("bits", [8, 4])
def test_cifar_network_small_batch(qnn, orc, bits):
    net = synth.cifar_network(bits=bits, n=5)
    check_network(qnn, orc, net)
    check_network(qnn, orc, net, fused=False)


@pytest.mark.parametrize("bits", [8, 4])
def test_cifar_network_batch4096(qnn, orc, bits):
    """The whole batch-4096 network: every layer's pooled output and the
    logits of every image against the oracle."""
    check_network(qnn, orc, synth.cifar_network(bits=bits, n=4096))


# ------------------------------------------------------ random small layers

@pytest.mark.parametrize("bits,epi", [(8, "requant"), (8, "raw32"), (4, "requant"),
                                      (4, "raw32"), (2, "requant"), (2, "raw32"),
                                      (1, "thresh1"), (1, "raw32")])
def test_random_layers(qnn, orc, bits, epi):
    rng = np.random.default_rng(1000 + bits * 7 + len(epi))
    for _ in range(20):
        L = synth.random_small_layer(rng, bits, epi=epi)
        check_layer(orc, L)


# ------------------------------------------------------ edge cases

def make(bits, n, h, w, c, m, k, stride=1, pad=1, epi=None, seed=5, shift=10):
    hi = (1 << bits) - 1
    if bits == 1:
        return synth.conv_layer("edge_int1", 1, n, h, w, c, m, k, pad, seed, None, None,
                                thresh_rng=(-20, 20), epi=epi, stride=stride)
    return synth.conv_layer("edge_int%d" % bits, bits, n, h, w, c, m, k, pad, seed, (0, hi),
                            (-(1 << (bits - 1)), (1 << (bits - 1)) - 1),
                            bias_rng=(-hi * 50, hi * 50), mult_rng=(1, 1 << 10), shift=shift,
                            clip=(0, hi), epi=epi, stride=stride)


@pytest.mark.parametrize("bits", [8, 4, 2, 1])
def test_ragged_channel_counts(qnn, orc, bits):
    unit = 32 // bits
    for m in (1, 3, 5, 15, 17, 31, 33, 65, 70, 129):
        check_layer(orc, make(bits, 2, 7, 9, unit, m, 3))


@pytest.mark.parametrize("bits", [8, 4, 2, 1])
def test_geometry_corners(qnn, orc, bits):
    unit = 32 // bits
    cases = [
        (1, 1, 1, unit, 8, 1, 1, 0),      # 1x1 image, 1x1 kernel
        (2, 1, 1, unit, 8, 3, 1, 1),      # 1x1 image, 3x3 kernel, all-padding halo
        (1, 2, 3, unit, 8, 5, 1, 2),      # kernel larger than the image
        (3, 13, 11, 2 * unit, 24, 3, 2, 1),  # stride 2, ragged tiles
        (2, 17, 9, unit, 16, 3, 3, 0),    # stride 3, no pad
        (1, 40, 70, unit, 16, 3, 1, 1),   # several tiles per image, ragged rows
        (2, 5, 5, 4 * unit, 8, 5, 1, 4),  # pad as large as the kernel - 1... and more
    ]
    for (n, h, w, c, m, k, s, p) in cases:
        check_layer(orc, make(bits, n, h, w, c, m, k, s, p))


@pytest.mark.parametrize("bits", [8, 4, 2])
def test_wide_filters(qnn, orc, bits):
    """Large C: long K walks and the multi-M-tile path."""
    c = {8: 256, 4: 256, 2: 512}[bits]
    check_layer(orc, make(bits, 2, 6, 6, c, 96, 3, shift=14))


@pytest.mark.parametrize("bits", [8, 4, 2])
def test_plan_extremes(qnn, orc, bits):
    """The largest shift the plans take (30) with small multipliers (threshold
    quotients up to 2^38: the floor divisions at the top of their range) and
    with multipliers just below 2^shift, and shift 24 with multipliers
    around 2^21, on the general kernels (pixels of two words and more)."""
    hi = (1 << bits) - 1
    unit = 32 // bits
    for j, (mult_rng, shift) in enumerate([((1, 1 << 8), 30), ((1 << 29, 1 << 30), 30),
                                           ((1 << 20, 1 << 22), 24)]):
        L = synth.conv_layer("plan_int%d" % bits, bits, 2, 9, 11, 2 * unit, 40, 3, 1, 60 + j, (0, hi),
                             (-(1 << (bits - 1)), (1 << (bits - 1)) - 1), bias_rng=(-hi * 50, hi * 50),
                             mult_rng=mult_rng, shift=shift, clip=(0, hi))
        check_layer(orc, L)


def test_batch_zero_launches_nothing(qnn):
    import torch
    x = torch.zeros((0, 4, 4, 4), dtype=torch.uint8, device="cuda")
    w = torch.zeros((8, 36), dtype=torch.uint8, device="cuda")
    y = qnn.conv2d(x, (0, 4, 4, 4), 8, w, 8, 3, 3, (1, 1), (1, 1), "raw32")
    assert y.shape == (0, 4, 4, 8)


def test_deterministic_and_stream_independent(qnn, orc):
    import torch
    L = synth.int4_layer(n=16)
    a = gpu_conv(L)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        b = gpu_conv(L, stream=s)
    c = gpu_conv(L)
    assert np.array_equal(a, b) and np.array_equal(a, c)


# ------------------------------------------------------ helpers

@pytest.mark.parametrize("bits", [8, 4, 2, 1])
def test_linear(qnn, orc, bits):
    import torch
    rng = np.random.default_rng(90 + bits)
    # K a multiple of 64 (the fully connected kernel) with ragged image and
    # channel counts, and K = 96 at 8 bits (the convolution tiles); 20 and 21
    # K steps of 64 run the four-step block and then the remainder loop
    for (n, h, w, c, m) in [(37, 4, 4, 64, 10), (5, 1, 1, 1024, 10), (9, 2, 3, 32 * 4 // bits, 33),
                            (300, 4, 4, 128, 70), (16, 1, 1, 4096, 16), (33, 8, 8, 64, 1),
                            (19, 1, 1, 64 * 20, 12), (19, 1, 1, 64 * 21, 10)]:
        if bits == 1:
            xv = 2 * rng.integers(0, 2, size=(n, h, w, c)) - 1
            wv = 2 * rng.integers(0, 2, size=(m, h * w * c)) - 1
        else:
            xv = rng.integers(0, 1 << bits, size=(n, h, w, c))
            wv = rng.integers(-(1 << (bits - 1)), 1 << (bits - 1), size=(m, h * w * c))
        x = synth.pack_codes(synth.to_code(xv, bits, False), bits)
        wt = synth.pack_codes(synth.to_code(wv, bits, True), bits)
        bias = rng.integers(-1000, 1000, size=m).astype(np.int32)
        # every other case without a bias (NULL: zero)
        if m % 2 == 0:
            bias = None
        log("case linear bits=%d n=%d k=%d m=%d bias=%s" % (bits, n, h * w * c, m, bias is not None))
        y = qnn.linear(dev(x), (n, h, w, c), bits, dev(wt), m, "raw32", bias=dev(bias))
        torch.cuda.synchronize()
        _, want = orc.linear(x.reshape(n, -1), n, h * w * c, bits, wt, m, epi=2,
                             bias=bias if bias is not None else np.zeros(m, np.int32))
        assert np.array_equal(y.cpu().numpy().reshape(n, m), want)


@pytest.mark.parametrize("bits", [8, 4, 2])
def test_maxpool(qnn, orc, bits):
    import torch
    rng = np.random.default_rng(80 + bits)
    for (n, h, w, c, k, s) in [(3, 32, 32, 32 * 8 // bits, 2, 2), (2, 9, 7, 4 * 8 // bits, 3, 2),
                               (1, 5, 5, 12 * 8 // bits, 1, 1), (4, 6, 8, 8 * 8 // bits, 2, 3)]:
        vals = rng.integers(0, 1 << bits, size=(n, h, w, c))
        x = synth.pack_codes(vals, bits)
        log("case maxpool bits=%d %s k=%d s=%d" % (bits, (n, h, w, c), k, s))
        y = qnn.maxpool2d(dev(x), (n, h, w, c), bits, k, k, s, s)
        torch.cuda.synchronize()
        assert np.array_equal(y.cpu().numpy(), orc.maxpool2d(x, (n, h, w, c), bits, k, k, s, s))


def test_relu_s8(qnn, orc):
    import torch
    rng = np.random.default_rng(3)
    for count in (1, 3, 4, 5, 255, 4096, 100003):
        x = rng.integers(-128, 128, size=count).astype(np.int8)
        xd = dev(x)
        y = qnn.relu_s8(xd)
        qnn.relu_s8(xd, out=xd)  # in place
        torch.cuda.synchronize()
        want = orc.relu_s8(x)
        assert np.array_equal(y.cpu().numpy(), want)
        assert np.array_equal(xd.cpu().numpy(), want)


def test_int1_register_resident_shapes(qnn, orc):
    """Filter volumes of 8..128 words take the register-resident XNOR path."""
    for (c, k, m) in [(256, 1, 40), (64, 2, 32), (256, 3, 64), (128, 4, 33), (512, 2, 70),
                      (1024, 1, 8), (256, 4, 32), (128, 5, 32)]:
        check_layer(orc, make(1, 2, 7, 6, c, m, k, pad=k // 2))


def test_int1_every_register_resident_volume(qnn, orc):
    """Every filter volume the register-resident XNOR kernel is built for
    (8..128 words in steps of 8), through the quad-wide im2col gather
    (channel words a multiple of 4) and the word-by-word one, with binary
    threshold and raw outputs."""
    cases = [(256 * j, 1) for j in range(1, 17)]            # 1x1 filters, 8j words per pixel
    cases += [(64, 2), (192, 2), (64, 4), (320, 2), (64, 6), (96, 4)]  # 2 or 6 words per tap
    for i, (c, k) in enumerate(cases):
        L = make(1, 1, 5, 6, c, 40, k, pad=k // 2, seed=100 + i)
        check_layer(orc, L)
        check_layer(orc, L, epi="raw32")
