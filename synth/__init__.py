"""Seeded synthetic workloads for the quantized convolution layer.

This module only draws random integer codes and lays them out in the stored
format of the layer's tensors (NHWC activations, OHWI weights, sub-byte codes
packed with the lower channel in the less significant bits, pixels padded to
whole bytes with zero bits).  It holds none of the layer's arithmetic: no
accumulation, no requantization, no thresholding.  Both the CPU oracle and the
GPU library consume the arrays it returns.

Generator: numpy PCG64, ``default_rng(seed).integers(lo, hi, size,
endpoint=True, dtype=int64)``; draw order per workload is fixed (input,
weights, bias, multiplier, threshold; for the CIFAR-shaped network: input,
then per layer weights, bias, multiplier, then the classifier's weights and
bias).  The workloads take the shapes and value ranges of the paper's layers:
the 16x16x32 -> 64 benchmark layer of Sec. V-A and the CIFAR-10 network of
Sec. V-E (synthetic images stand in for the dataset; weights are random).
"""
from dataclasses import dataclass, field
import hashlib

import numpy as np


def pack_codes(codes, bits):
    """Lay out unsigned codes (last axis = elements of one pixel/row) in the
    packed storage format.  bits in {1, 2, 4, 8}; the last axis is padded to
    whole bytes with zero bits."""
    codes = np.asarray(codes, dtype=np.int64)
    if codes.size and (codes.min() < 0 or codes.max() >= (1 << bits)):
        raise ValueError("code out of range for %d bits" % bits)
    per = 8 // bits
    lead = codes.shape[:-1]
    c = codes.shape[-1]
    nbytes = (c * bits + 7) // 8
    padded = np.zeros(lead + (nbytes * per,), dtype=np.int64)
    padded[..., :c] = codes
    grouped = padded.reshape(lead + (nbytes, per))
    out = np.zeros(lead + (nbytes,), dtype=np.int64)
    for j in range(per):
        out |= grouped[..., j] << (j * bits)
    return out.astype(np.uint8)


def to_code(values, bits, signed):
    """Integer value -> stored code: two's complement for signed 8/4/2-bit
    weights, identity for unsigned activations, (v + 1) / 2 for +-1 values."""
    v = np.asarray(values, dtype=np.int64)
    if bits == 1:
        return (v + 1) // 2
    if signed:
        return v & ((1 << bits) - 1)
    return v


def sha256(*arrays):
    h = hashlib.sha256()
    for a in arrays:
        if a is not None:
            h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


@dataclass
class ConvLayer:
    """One quantized convolution layer: packed tensors plus the integer
    values they encode (for the tests' independent references)."""
    name: str
    bits: int
    n: int
    h: int
    w: int
    c: int
    m: int
    kh: int
    kw: int
    stride: tuple
    pad: tuple
    epi: str                      # "requant" | "thresh1" | "raw32"
    x_vals: np.ndarray            # int64 [N,H,W,C]  activation values
    w_vals: np.ndarray            # int64 [M,kh,kw,C] weight values
    bias: np.ndarray = None       # int32 [M]
    mult: np.ndarray = None       # int32 [M]
    shift: np.ndarray = None      # int8  [M]
    thresh: np.ndarray = None     # int32 [M]
    clip: tuple = (0, 0)
    c_alg: int = 0                # channels that carry data (MAC count)
    x: np.ndarray = field(init=False)   # uint8 packed [N,H,W,Pb]
    wt: np.ndarray = field(init=False)  # uint8 packed [M, kh*kw*C bytes]

    def __post_init__(self):
        if self.c_alg == 0:
            self.c_alg = self.c
        self.x = pack_codes(to_code(self.x_vals, self.bits, signed=False), self.bits)
        wcodes = to_code(self.w_vals, self.bits, signed=True).reshape(self.m, -1)
        self.wt = pack_codes(wcodes, self.bits)

    @property
    def ho(self):
        return (self.h + 2 * self.pad[0] - self.kh) // self.stride[0] + 1

    @property
    def wo(self):
        return (self.w + 2 * self.pad[1] - self.kw) // self.stride[1] + 1

    @property
    def macs(self):
        """Dense MAC count: every output element times the filter volume,
        padded taps included; channels added only for alignment excluded."""
        return self.n * self.ho * self.wo * self.m * self.kh * self.kw * self.c_alg

    def digest(self):
        return sha256(self.x, self.wt, self.bias, self.mult, self.shift, self.thresh)


def _draw(rng, lo, hi, size):
    return rng.integers(lo, hi, size=size, endpoint=True, dtype=np.int64)


def _bits_draw(rng, size):
    """+-1 values, each drawn as a fair bit."""
    return 2 * rng.integers(0, 1, size=size, endpoint=True, dtype=np.int64) - 1


def conv_layer(name, bits, n, h, w, c, m, k, pad, seed, x_rng, w_rng, bias_rng=None,
               mult_rng=(1 << 14, 1 << 15), shift=None, clip=None, thresh_rng=None, epi=None,
               stride=1, stair_sorted=True):
    """Draw one layer's tensors in the fixed order x, w, bias, mult, thresh.

    epi "stair" draws 2^bits - 1 thresholds per channel from thresh_rng,
    sorted per channel unless stair_sorted is False."""
    rng = np.random.default_rng(seed)
    if bits == 1:
        x_vals = _bits_draw(rng, (n, h, w, c))
        w_vals = _bits_draw(rng, (m, k, k, c))
    else:
        x_vals = _draw(rng, x_rng[0], x_rng[1], (n, h, w, c))
        w_vals = _draw(rng, w_rng[0], w_rng[1], (m, k, k, c))
    bias = _draw(rng, bias_rng[0], bias_rng[1], m).astype(np.int32) if bias_rng else None
    mult = shiftv = thresh = None
    if epi is None:
        epi = "thresh1" if bits == 1 else "requant"
    if epi == "requant":
        mult = _draw(rng, mult_rng[0], mult_rng[1], m).astype(np.int32)
        shiftv = np.full(m, shift, dtype=np.int8)
    if bits == 1 and thresh_rng is not None:
        thresh = _draw(rng, thresh_rng[0], thresh_rng[1], m).astype(np.int32)
    if epi == "stair":
        thresh = _draw(rng, thresh_rng[0], thresh_rng[1], (m, (1 << bits) - 1)).astype(np.int32)
        if stair_sorted:
            thresh = np.sort(thresh, axis=1)
    return ConvLayer(name, bits, n, h, w, c, m, k, k, (stride, stride), (pad, pad), epi, x_vals,
                     w_vals, bias, mult, shiftv, thresh, clip or (0, 0))


# --- the single-layer workloads -------------------------------------------

def int8_layer(n=1):
    """INT8 3x3 layer on a 16x16x32 input, 32 filters (benchmark layer of
    Sec. V-A with 32 output channels)."""
    return conv_layer("int8_16x16x32_m32_b%d" % n, 8, n, 16, 16, 32, 32, 3, 1, seed=0,
                      x_rng=(0, 255), w_rng=(-128, 127), bias_rng=(-4096, 4096), shift=22,
                      clip=(0, 255))


def int4_layer(n=64):
    """INT4 3x3 layer, 32x32x64 input, 64 filters."""
    return conv_layer("int4_32x32x64_m64_b%d" % n, 4, n, 32, 32, 64, 64, 3, 1, seed=1,
                      x_rng=(0, 15), w_rng=(-8, 7), bias_rng=(-256, 256), shift=21,
                      clip=(0, 15))


def headline_shape_layer(bits, n=64):
    """The INT4 layer's shape (3x3, 32x32x64 input, 64 filters, batch n) at
    8, 4 or 2 bits, for comparing tile shapes across bit-widths."""
    if bits == 4:
        return int4_layer(n)
    hi, wlo = (1 << bits) - 1, -(1 << (bits - 1))
    return conv_layer("int%d_32x32x64_m64_b%d" % (bits, n), bits, n, 32, 32, 64, 64, 3, 1,
                      seed=10 + bits, x_rng=(0, hi), w_rng=(wlo, -wlo - 1),
                      bias_rng=(-16 * hi, 16 * hi), shift={8: 23, 2: 19}[bits], clip=(0, hi))


def int4_stair_layer(n=64):
    """The INT4 layer's shape and seed with the staircase epilogue of
    Sec. III-A, Eq. (4): 15 sorted thresholds per channel drawn from
    U[-15120, 15120] (a quarter of K * max x * max w)."""
    return conv_layer("int4_stair_32x32x64_m64_b%d" % n, 4, n, 32, 32, 64, 64, 3, 1, seed=1,
                      x_rng=(0, 15), w_rng=(-8, 7), bias_rng=(-256, 256),
                      thresh_rng=(-15120, 15120), epi="stair")


def int2_layer(n=256):
    """INT2 3x3 layer, 16x16x128 input, 128 filters."""
    return conv_layer("int2_16x16x128_m128_b%d" % n, 2, n, 16, 16, 128, 128, 3, 1, seed=2,
                      x_rng=(0, 3), w_rng=(-2, 1), bias_rng=(-64, 64), shift=20, clip=(0, 3))


def int1_layer(n=1024):
    """INT1 (binary) 3x3 layer, 8x8x256 input, 256 filters, one threshold per
    output channel."""
    return conv_layer("int1_8x8x256_m256_b%d" % n, 1, n, 8, 8, 256, 256, 3, 1, seed=3,
                      x_rng=None, w_rng=None, thresh_rng=(-128, 128))


def centred(layer):
    """Same tensors, with the bias shifted so that a typical accumulator lands
    mid-range: bias_m - floor(hi * sum_k w[m,k] / 2).  Used to exercise every
    output code of the sub-byte layers (whose literal bias ranges leave almost
    every output at zero)."""
    hi = layer.clip[1]
    wsum = layer.w_vals.reshape(layer.m, -1).sum(axis=1)
    bias = (layer.bias.astype(np.int64) - np.floor_divide(hi * wsum, 2)).astype(np.int32)
    out = ConvLayer(layer.name + "_centred", layer.bits, layer.n, layer.h, layer.w, layer.c,
                    layer.m, layer.kh, layer.kw, layer.stride, layer.pad, layer.epi,
                    layer.x_vals, layer.w_vals, bias, layer.mult, layer.shift, layer.thresh,
                    layer.clip, layer.c_alg)
    return out


# --- the CIFAR-10-shaped network (Sec. V-E shapes) ------------------------

@dataclass
class Network:
    name: str
    bits: int
    n: int
    x_vals: np.ndarray       # [N,32,32,Cpad]
    c_alg: int               # 3 image channels
    convs: list              # per conv: dict(w_vals, bias, mult, shift, m, k, pad)
    fc_w_vals: np.ndarray    # [10, 1024]
    fc_bias: np.ndarray
    clip: tuple

    def packed_input(self):
        return pack_codes(to_code(self.x_vals, self.bits, False), self.bits)


def cifar_network(bits=8, n=4096, seed=4):
    """Three 5x5 conv layers (3->32, 32->32, 32->64, pad 2, requant + ReLU clip,
    2x2 max-pool after each) and a 1024->10 classifier with int32 logits.

    The 3 image channels are padded with a zero channel (and zero weights) to
    4 channels: a pixel of 4 bytes at 8 bits, of 2 bytes at 4 bits."""
    rng = np.random.default_rng(seed)
    if bits == 8:
        xr, wr, br, shift, clip, cpad = (0, 255), (-128, 127), (-4096, 4096), 25, (0, 255), 4
    elif bits == 4:
        xr, wr, br, shift, clip, cpad = (0, 15), (-7, 7), (-256, 256), 21, (0, 15), 4
    else:
        raise ValueError("CIFAR-shaped network is defined at 8 and 4 bits")
    x3 = _draw(rng, xr[0], xr[1], (n, 32, 32, 3))
    x = np.zeros((n, 32, 32, cpad), dtype=np.int64)
    x[..., :3] = x3
    convs = []
    cin, cin_pad = 3, cpad
    for m in (32, 32, 64):
        w_alg = _draw(rng, wr[0], wr[1], (m, 5, 5, cin))
        wv = np.zeros((m, 5, 5, cin_pad), dtype=np.int64)
        wv[..., :cin] = w_alg
        bias = _draw(rng, br[0], br[1], m).astype(np.int32)
        mult = _draw(rng, 1 << 14, 1 << 15, m).astype(np.int32)
        convs.append(dict(w_vals=wv, bias=bias, mult=mult, shift=np.full(m, shift, np.int8),
                          m=m, k=5, pad=2, c=cin_pad, c_alg=cin))
        cin = cin_pad = m
    fc_w = _draw(rng, wr[0], wr[1], (10, 4 * 4 * 64))
    fc_b = _draw(rng, br[0], br[1], 10).astype(np.int32)
    return Network("cifar_int%d_b%d" % (bits, n), bits, n, x, 3, convs, fc_w, fc_b, clip)


def network_macs(net):
    """Dense MACs of the CIFAR-shaped network per batch (padding channels
    excluded)."""
    macs = 0
    hw = 32
    for cv in net.convs:
        macs += net.n * hw * hw * cv["m"] * 25 * cv["c_alg"]
        hw //= 2
    macs += net.n * net.fc_w_vals.size
    return macs


def random_small_layer(rng, bits, epi=None):
    """A small random layer for parity sweeps: ragged spatial sizes, strides
    1-2, pads 0-2, kernels 1-5, channel counts that fill whole 4-byte pixels."""
    unit = 32 // bits  # channels per 4 bytes
    c = unit * int(rng.integers(1, 4))
    m = int(rng.integers(1, 80 if bits == 1 else 41))
    k = int(rng.choice([1, 3, 5]))
    stride = int(rng.integers(1, 3))
    pad = int(rng.integers(0, 3))
    h = int(rng.integers(max(1, k - 2 * pad), 12))
    w = int(rng.integers(max(1, k - 2 * pad), 12))
    n = int(rng.integers(1, 4))
    seed = int(rng.integers(0, 2**31))
    if bits == 1:
        return conv_layer("rand_int1", 1, n, h, w, c, m, k, pad, seed, None, None,
                          bias_rng=None, thresh_rng=(-k * k * c, k * k * c), epi=epi,
                          stride=stride)
    hi = (1 << bits) - 1
    wlo, whi = -(1 << (bits - 1)), (1 << (bits - 1)) - 1
    span = max(1, k * k * c * hi * whi // 4)  # thresholds of "stair" layers
    return conv_layer("rand_int%d" % bits, bits, n, h, w, c, m, k, pad, seed, (0, hi),
                      (wlo, whi), bias_rng=(-hi * 64, hi * 64), shift=int(rng.integers(8, 16)),
                      clip=(0, hi), epi=epi, stride=stride, thresh_rng=(-span, span))
