"""Pins of the CPU oracle to things other than itself (CPU only).

Each test names what fixes the expected value:
  * a library routine (torch float64 conv2d / max_pool2d / matmul, exact on
    these integer sizes);
  * a brute-force evaluator written separately with Python integers;
  * closed forms and invariants (identity and one-hot filters, linearity, the
    INT-1 XNOR/popcount identity of Sec. III-A Eq. (5), the staircase of
    Sec. III-A Eq. (4) that scale-and-clamp must equal);
  * hand-worked values stored under tests/golden/ with their citation.
"""
import bisect
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
EPI = {"requant": 0, "thresh1": 1, "raw32": 2, "stair": 3}


def golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield [p.strip() for p in line.split("|")]


def run_oracle(orc, L, want_acc=True, want_y=True, nthreads=1):
    return orc.conv2d(L.x, (L.n, L.h, L.w, L.c), L.bits, L.wt, L.m, L.kh, L.kw, L.stride, L.pad,
                      EPI[L.epi], L.bias, L.mult, L.shift, L.thresh, L.clip, want_acc=want_acc,
                      want_y=want_y, nthreads=nthreads)


def torch_conv_f64(x_vals, w_vals, stride, pad, pad_value):
    """Eq. (6) through a library routine: float64 cross-correlation, exact for
    |acc| < 2^53."""
    x = torch.tensor(x_vals, dtype=torch.float64).permute(0, 3, 1, 2)
    x = F.pad(x, (pad[1], pad[1], pad[0], pad[0]), value=float(pad_value))
    w = torch.tensor(w_vals, dtype=torch.float64).permute(0, 3, 1, 2)
    out = F.conv2d(x, w, stride=tuple(stride))
    return out.permute(0, 2, 3, 1).numpy().astype(np.int64)


def random_layers(bits, count, seed, epi=None):
    rng = np.random.default_rng(seed)
    return [synth.random_small_layer(rng, bits, epi=epi) for _ in range(count)]


# ---------------------------------------------------------------- P4 packing

def test_generator_packer_matches_golden():
    for bits, codes, hexbytes in golden_lines("packing_examples.txt"):
        codes = np.array([int(c) for c in codes.split()], dtype=np.int64)
        want = np.array([int(b, 16) for b in hexbytes.split()], dtype=np.uint8)
        got = synth.pack_codes(codes[None, :], int(bits))[0]
        assert np.array_equal(got, want), (bits, codes, got)


def test_oracle_pack_and_decode_match_golden(orc):
    for bits, codes, hexbytes in golden_lines("packing_examples.txt"):
        bits = int(bits)
        codes = np.array([int(c) for c in codes.split()], dtype=np.int64)
        packed = np.array([int(b, 16) for b in hexbytes.split()], dtype=np.uint8)
        assert np.array_equal(orc.pack(codes, bits), packed)
        vals = orc.unpack(packed, codes.size, bits, signed=False)
        want = 2 * codes - 1 if bits == 1 else codes
        assert np.array_equal(vals, want)


def test_sign_tables_match_golden(orc):
    for bits, values in golden_lines("sign_tables.txt"):
        bits = int(bits)
        values = [int(v) for v in values.split()]
        codes = np.arange(1 << bits)
        packed = synth.pack_codes(codes[None, :], bits)[0]
        assert list(orc.unpack(packed, codes.size, bits, signed=True)) == values
        # the generator's value -> code map is the inverse
        assert list(synth.to_code(np.array(values), bits, signed=True)) == list(codes)
    # 8 bits: two's complement byte, as numpy's int8 view of the byte
    codes = np.arange(256)
    got = orc.unpack(codes.astype(np.uint8), 256, 8, signed=True)
    assert np.array_equal(got, codes.astype(np.uint8).view(np.int8))


@pytest.mark.parametrize("bits", [1, 2, 4, 8])
def test_pack_roundtrip_random(orc, bits):
    rng = np.random.default_rng(bits)
    for count in (1, 7, 8, 9, 31, 64, 1000):
        codes = rng.integers(0, 1 << bits, size=count)
        packed = synth.pack_codes(codes[None, :], bits)[0]
        assert packed.size == (count * bits + 7) // 8
        assert np.array_equal(orc.pack(codes, bits), packed)
        vals = orc.unpack(packed, count, bits, signed=False)
        assert np.array_equal(vals, 2 * codes - 1 if bits == 1 else codes)
        # unused high bits of the last byte are zero
        tail = count * bits % 8
        if tail:
            assert packed[-1] >> tail == 0
        # bytes -> codes -> bytes
        anyb = rng.integers(0, 256, size=(count * bits + 7) // 8).astype(np.uint8)
        if tail:
            anyb[-1] &= (1 << tail) - 1
        dec = orc.unpack(anyb, count, bits, signed=False)
        dec_codes = (dec + 1) // 2 if bits == 1 else dec
        assert np.array_equal(orc.pack(dec_codes, bits), anyb)


# ------------------------------------------------- P1 library routine (f64)

@pytest.mark.parametrize("bits", [8, 4, 2, 1])
def test_accumulator_matches_torch_conv2d(orc, bits):
    for L in random_layers(bits, 12, seed=100 + bits):
        acc, _ = run_oracle(orc, L, want_y=False)
        ref = torch_conv_f64(L.x_vals, L.w_vals, L.stride, L.pad, -1 if bits == 1 else 0)
        assert acc.shape == ref.shape
        assert np.array_equal(acc, ref), L.name


def test_int8_benchmark_layer_matches_torch(orc):
    L = synth.int8_layer()
    acc, _ = run_oracle(orc, L, want_y=False)
    assert np.array_equal(acc, torch_conv_f64(L.x_vals, L.w_vals, L.stride, L.pad, 0))


def test_cifar_first_layer_matches_torch(orc):
    net = synth.cifar_network(bits=8, n=2)
    cv = net.convs[0]
    L = synth.ConvLayer("c", 8, 2, 32, 32, cv["c"], cv["m"], 5, 5, (1, 1), (2, 2), "raw32",
                        net.x_vals, cv["w_vals"], cv["bias"], c_alg=3)
    acc, _ = run_oracle(orc, L, want_y=False)
    assert np.array_equal(acc, torch_conv_f64(net.x_vals, cv["w_vals"], (1, 1), (2, 2), 0))


def test_padding_channels_change_nothing(orc):
    """Zero channels with zero weights (used to fill 4-byte pixels) leave the
    accumulator of the 3-channel layer unchanged."""
    net = synth.cifar_network(bits=8, n=1)
    cv = net.convs[0]
    full = synth.ConvLayer("p", 8, 1, 32, 32, 4, 32, 5, 5, (1, 1), (2, 2), "raw32", net.x_vals,
                           cv["w_vals"])
    three = synth.ConvLayer("t", 8, 1, 32, 32, 3, 32, 5, 5, (1, 1), (2, 2), "raw32",
                            net.x_vals[..., :3], cv["w_vals"][..., :3])
    a4, _ = run_oracle(orc, full, want_y=False)
    a3, _ = run_oracle(orc, three, want_y=False)
    assert np.array_equal(a4, a3)


# --------------------------------------------------- P2 brute force (ints)

def bf_code(pixel_bytes, i, bits):
    word = int.from_bytes(bytes(pixel_bytes), "little")
    return (word >> (i * bits)) & ((1 << bits) - 1)


def bf_value(code, bits, signed):
    if bits == 1:
        return 1 if code else -1
    if signed and code >> (bits - 1):
        return code - (1 << bits)
    return code


def brute_force(L):
    """Separately written evaluator: Python ints, whole-pixel integer decode."""
    pb = (L.c * L.bits + 7) // 8
    wb = (L.kh * L.kw * L.c * L.bits + 7) // 8
    xs = L.x.reshape(L.n, L.h, L.w, pb)
    ws = L.wt.reshape(L.m, wb)
    obits = {"requant": L.bits, "thresh1": 1, "raw32": 32, "stair": L.bits}[L.epi]
    out = []
    for n in range(L.n):
        for oy in range(L.ho):
            for ox in range(L.wo):
                word = 0
                for m in range(L.m):
                    acc = 0
                    for ky in range(L.kh):
                        for kx in range(L.kw):
                            iy = oy * L.stride[0] - L.pad[0] + ky
                            ix = ox * L.stride[1] - L.pad[1] + kx
                            for c in range(L.c):
                                if 0 <= iy < L.h and 0 <= ix < L.w:
                                    xv = bf_value(bf_code(xs[n, iy, ix], c, L.bits), L.bits, False)
                                else:
                                    xv = bf_value(0, L.bits, False)
                                k = (ky * L.kw + kx) * L.c + c
                                wv = bf_value(bf_code(ws[m], k, L.bits), L.bits, True)
                                acc += xv * wv
                    b = int(L.bias[m]) if L.bias is not None else 0
                    v = acc + b
                    if L.epi == "requant":
                        s = int(L.shift[m])
                        t = v * int(L.mult[m])
                        r = t if s == 0 else (t + (1 << (s - 1))) // (1 << s)
                        code = min(max(r, L.clip[0]), L.clip[1])
                    elif L.epi == "thresh1":
                        code = 1 if v >= int(L.thresh[m]) else 0
                    elif L.epi == "stair":
                        # sorted thresholds: the level is how many lie at or below v
                        code = bisect.bisect_right([int(t) for t in L.thresh[m]], v)
                    else:
                        code = v % (1 << 32)
                    word |= code << (m * obits)
                nbytes = L.m * 4 if obits == 32 else (L.m * obits + 7) // 8
                out.append(np.frombuffer(word.to_bytes(nbytes, "little"), dtype=np.uint8))
    return np.stack(out)


def tiny_layers(bits, count, seed, epi):
    rng = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        L = synth.random_small_layer(rng, bits, epi=epi)
        if L.n * L.ho * L.wo * L.m * L.kh * L.kw * L.c <= 60000:
            out.append(L)
    return out


@pytest.mark.parametrize("bits,epi", [(8, "requant"), (4, "requant"), (2, "requant"),
                                      (8, "raw32"), (4, "raw32"), (2, "raw32"), (1, "raw32"),
                                      (1, "thresh1"), (4, "stair"), (2, "stair")])
def test_oracle_matches_brute_force(orc, bits, epi):
    for L in tiny_layers(bits, 4, seed=200 + bits + len(epi), epi=epi):
        _, y = run_oracle(orc, L, want_acc=False)
        got = y.reshape(L.n * L.ho * L.wo, -1).view(np.uint8)
        assert np.array_equal(got, brute_force(L)), L.name


def test_requant_spread_brute_force(orc):
    """A tiny layer whose outputs cover 0, the clip top and values in between."""
    rng = np.random.default_rng(7)
    L = synth.conv_layer("spread", 4, 2, 5, 5, 8, 6, 3, 1, seed=11, x_rng=(0, 15),
                         w_rng=(-8, 7), bias_rng=(-300, 300), mult_rng=(1, 2), shift=5,
                         clip=(0, 15))
    _, y = run_oracle(orc, L)
    got = y.reshape(L.n * L.ho * L.wo, -1)
    assert np.array_equal(got, brute_force(L))
    codes = np.concatenate([(got & 15).ravel(), (got >> 4).ravel()])
    assert (codes == 0).any() and (codes == 15).any() and ((codes > 0) & (codes < 15)).any()
    del rng


# ------------------------------------------------- P3 identity and one-hot

@pytest.mark.parametrize("bits", [8, 4, 2])
def test_identity_filter_returns_input(orc, bits):
    hi = (1 << bits) - 1
    c = 4 * (8 // bits)
    rng = np.random.default_rng(bits)
    x_vals = rng.integers(0, hi + 1, size=(2, 5, 7, c))
    w_vals = np.eye(c, dtype=np.int64).reshape(c, 1, 1, c)
    L = synth.ConvLayer("id", bits, 2, 5, 7, c, c, 1, 1, (1, 1), (0, 0), "requant", x_vals,
                        w_vals, np.zeros(c, np.int32), np.ones(c, np.int32), np.zeros(c, np.int8),
                        None, (0, hi))
    _, y = run_oracle(orc, L)
    assert np.array_equal(y, L.x)


@pytest.mark.parametrize("bits", [8, 4, 2])
def test_one_hot_filter_shifts_input(orc, bits):
    hi = (1 << bits) - 1
    c = 4 * (8 // bits)
    rng = np.random.default_rng(10 + bits)
    x_vals = rng.integers(0, hi + 1, size=(1, 6, 5, c))
    for a in range(3):
        for b in range(3):
            w_vals = np.zeros((c, 3, 3, c), dtype=np.int64)
            for m in range(c):
                w_vals[m, a, b, m] = 1
            L = synth.ConvLayer("oh", bits, 1, 6, 5, c, c, 3, 3, (1, 1), (1, 1), "requant",
                                x_vals, w_vals, np.zeros(c, np.int32), np.ones(c, np.int32),
                                np.zeros(c, np.int8), None, (0, hi))
            _, y = run_oracle(orc, L)
            want = np.zeros_like(x_vals)
            for oy in range(6):
                for ox in range(5):
                    iy, ix = oy - 1 + a, ox - 1 + b
                    if 0 <= iy < 6 and 0 <= ix < 5:
                        want[0, oy, ox] = x_vals[0, iy, ix]
            assert np.array_equal(y, synth.pack_codes(want, bits)), (a, b)


# ------------------------------------------- P5 INT-1 XNOR/popcount identity

def xnor_popcount_dot(L):
    """Eq. (5): popcount(W xnor X) over the receptive field, pad bits 0, then
    dot = 2 * popcount - K.  Works on the packed bits directly."""
    xb = np.unpackbits(L.x, axis=-1, bitorder="little")[..., :L.c]
    wb = np.unpackbits(L.wt, axis=-1, bitorder="little")[:, :L.kh * L.kw * L.c]
    wb = wb.reshape(L.m, L.kh, L.kw, L.c)
    xp = np.zeros((L.n, L.h + 2 * L.pad[0], L.w + 2 * L.pad[1], L.c), dtype=np.uint8)
    xp[:, L.pad[0]:L.pad[0] + L.h, L.pad[1]:L.pad[1] + L.w] = xb
    K = L.kh * L.kw * L.c
    out = np.zeros((L.n, L.ho, L.wo, L.m), dtype=np.int64)
    for oy in range(L.ho):
        for ox in range(L.wo):
            y0, x0 = oy * L.stride[0], ox * L.stride[1]
            field = xp[:, y0:y0 + L.kh, x0:x0 + L.kw, :].reshape(L.n, 1, K)
            xn = 1 - (field ^ wb.reshape(1, L.m, K))
            out[:, oy, ox, :] = 2 * xn.sum(axis=-1) - K
    return out


def test_int1_xnor_popcount_equals_pm1_dot(orc):
    layers = random_layers(1, 10, seed=300) + [synth.int1_layer(n=2)]
    for L in layers:
        acc, _ = run_oracle(orc, L, want_y=False)
        assert np.array_equal(acc, xnor_popcount_dot(L)), L.name


# --------------------------------- P6 scale-and-clamp = staircase (Eq. (4))

def test_requant_equals_threshold_staircase(orc):
    """For mult > 0 the rounding right shift followed by the clip is the
    staircase of Eq. (4) with 2^Q - 1 thresholds:
        y = #{p in 1..hi : acc + bias >= ceil((p 2^(s+1) - 2^s) / (2 mult))}."""
    rng = np.random.default_rng(5)
    # acc = u + 127 v over a contiguous range via a 2-input linear layer
    u = np.arange(0, 127)
    v = np.arange(0, 256, 3)
    uu, vv = np.meshgrid(u, v)
    x = np.stack([uu.ravel(), vv.ravel()], axis=1)
    n = x.shape[0]
    acc = x[:, 0] + 127 * x[:, 1]
    m = 24
    wt = synth.pack_codes(synth.to_code(np.tile([[1, 127]], (m, 1)), 8, True), 8)
    mult = rng.integers(1, 1 << 15, size=m).astype(np.int32)
    shift = rng.integers(0, 24, size=m).astype(np.int8)
    bias = rng.integers(-40000, 8000, size=m).astype(np.int32)
    for bits in (8,):
        hi = (1 << bits) - 1
        _, y = orc.linear(synth.pack_codes(x, 8), n, 2, 8, wt, m, epi=0, bias=bias, mult=mult,
                          shift=shift, clip=(0, hi))
        for j in range(m):
            s, M, b = int(shift[j]), int(mult[j]), int(bias[j])
            taus = [-(-(p * (1 << (s + 1)) - (1 << s)) // (2 * M)) - b for p in range(1, hi + 1)]
            stair = (acc[:, None] >= np.array(taus)[None, :]).sum(axis=1)
            assert np.array_equal(y[:, j].astype(np.int64), stair), j


def staircase_from_requant(bias, mult, shift, bits):
    """Thresholds on acc (bias folded in) that reproduce scale-and-clamp with
    clip (0, 2^bits - 1): level p is reached once (acc + b) mult + 2^(s-1) >=
    p 2^s, i.e. acc >= ceil((p 2^s - 2^(s-1)) / mult) - b."""
    m = len(bias)
    nt = (1 << bits) - 1
    tau = np.zeros((m, nt), dtype=np.int64)
    for j in range(m):
        s, M, b = int(shift[j]), int(mult[j]), int(bias[j])
        half = (1 << (s - 1)) if s else 0
        for p in range(1, nt + 1):
            tau[j, p - 1] = -((half - p * (1 << s)) // M) - b
    return tau


@pytest.mark.parametrize("bits", [4, 2])
def test_stair_equals_requant_with_derived_thresholds(orc, bits):
    """The staircase epilogue (Eq. (4)) fed with the thresholds of a
    multiplier/shift compression gives the same codes as scale-and-clamp."""
    rng = np.random.default_rng(60 + bits)
    hi = (1 << bits) - 1
    count = 0
    for L in tiny_layers(bits, 6, seed=70 + bits, epi="requant"):
        L.clip = (0, hi)
        _, want = run_oracle(orc, L, want_acc=False)
        tau = staircase_from_requant(L.bias, L.mult, L.shift, bits)
        if np.abs(tau).max() >= 1 << 31:
            continue
        _, got = orc.conv2d(L.x, (L.n, L.h, L.w, L.c), bits, L.wt, L.m, L.kh, L.kw, L.stride, L.pad,
                            EPI["stair"], None, None, None, tau.astype(np.int32), (0, 0))
        assert np.array_equal(got, want), L.name
        count += 1
    assert count >= 3
    del rng


@pytest.mark.parametrize("bits", [4, 2])
def test_stair_unsorted_thresholds_count(orc, bits):
    """Unsorted thresholds: the code is the number of thresholds at or below
    acc + bias (checked by brute-force counting on the accumulators)."""
    rng = np.random.default_rng(90 + bits)
    L = synth.random_small_layer(rng, bits, epi="stair")
    L.thresh = np.ascontiguousarray(rng.permuted(L.thresh, axis=1))
    acc, y = run_oracle(orc, L)
    b = L.bias.astype(np.int64)
    phi = acc + b[None, None, None, :]
    cnt = (phi[..., None] >= L.thresh.astype(np.int64)[None, None, None, :, :]).sum(axis=-1)
    want = synth.pack_codes(cnt.reshape(-1, L.m), bits)
    assert np.array_equal(y.reshape(want.shape), want)


def test_hand_worked_stair(orc):
    x1 = np.array([[1]], dtype=np.uint8)
    for f in golden_lines("stair_examples.txt"):
        bits, phi = int(f[0]), int(f[1])
        tau = np.array([[int(t) for t in f[2].split(",")]], dtype=np.int32)
        want = int(f[3])
        # a 1-input linear layer with x = 1 and w = +1 (acc = 1, bias = phi - 1)
        # or w = -1 (acc = -1, bias = phi + 1), whichever keeps the bias in int32
        wcode = 1 if phi >= 0 else (1 << bits) - 1
        bias = phi - 1 if phi >= 0 else phi + 1
        _, y = orc.linear(x1, 1, 1, bits, np.array([[wcode]], dtype=np.uint8), 1, epi=EPI["stair"],
                          bias=np.array([bias]), thresh=tau)
        assert int(y[0, 0]) == want, f


# ----------------------------------------------- P7 hand-worked examples

def test_hand_worked_requant_and_threshold(orc):
    x0 = np.zeros((1, 1), dtype=np.uint8)
    w0 = np.zeros((1, 1), dtype=np.uint8)
    for f in golden_lines("requant_examples.txt"):
        if f[0] == "requant":
            v, mult, shift, lo, hi, want = map(int, f[1:])
            _, y = orc.linear(x0, 1, 1, 8, w0, 1, epi=0, bias=np.array([v]),
                              mult=np.array([mult]), shift=np.array([shift]), clip=(lo, hi))
            assert int(y[0, 0]) == want, f
        else:
            dot, th, want = map(int, f[1:])
            # one +1 * +1 product (dot 1) plus a bias of dot - 1
            xb = np.array([[1]], dtype=np.uint8)
            wb = np.array([[1]], dtype=np.uint8)
            _, y = orc.linear(xb, 1, 1, 1, wb, 1, epi=1, bias=np.array([dot - 1]),
                              thresh=np.array([th]))
            assert int(y[0, 0]) == want, f


# ---------------------------------------------------------- P8 linearity

@pytest.mark.parametrize("bits", [8, 4, 2])
def test_linearity_in_weights(orc, bits):
    rng = np.random.default_rng(40 + bits)
    half = {8: (-64, 63), 4: (-4, 3), 2: (-1, 0)}[bits]
    hi = (1 << bits) - 1
    c = 2 * (32 // bits)
    x_vals = rng.integers(0, hi + 1, size=(2, 7, 6, c))
    w1 = rng.integers(half[0], half[1] + 1, size=(5, 3, 3, c))
    w2 = rng.integers(half[0], half[1] + 1, size=(5, 3, 3, c))
    accs = []
    for wv in (w1, w2, w1 + w2):
        L = synth.ConvLayer("lin", bits, 2, 7, 6, c, 5, 3, 3, (1, 1), (1, 1), "raw32", x_vals, wv)
        accs.append(run_oracle(orc, L, want_y=False)[0])
    assert np.array_equal(accs[0] + accs[1], accs[2])


# ---------------------------------------------------- P9 INT-8 sign fold

def test_int8_offset_identity(orc):
    """sum x*w = sum (x - 128)*w + 128 * sum w, with padding taps at x = 0
    (the unsigned-to-signed fold the GPU kernels use)."""
    L = synth.int8_layer()
    acc, _ = run_oracle(orc, L, want_y=False)
    shifted = torch_conv_f64(L.x_vals - 128, L.w_vals, L.stride, L.pad, -128)
    wsum = L.w_vals.reshape(L.m, -1).sum(axis=1)
    assert np.array_equal(acc, shifted + 128 * wsum[None, None, None, :])


# ------------------------------------------------------------ P10 helpers

@pytest.mark.parametrize("bits", [8, 4, 2])
def test_maxpool_matches_torch(orc, bits):
    rng = np.random.default_rng(60 + bits)
    hi = (1 << bits) - 1
    for (h, w, k, s) in [(8, 8, 2, 2), (7, 9, 2, 2), (9, 5, 3, 2), (6, 6, 3, 3), (5, 4, 1, 1)]:
        c = 3 * (32 // bits)
        vals = rng.integers(0, hi + 1, size=(2, h, w, c))
        y = orc.maxpool2d(synth.pack_codes(vals, bits), (2, h, w, c), bits, k, k, s, s)
        ref = F.max_pool2d(torch.tensor(vals, dtype=torch.float64).permute(0, 3, 1, 2), k, s)
        ref = ref.permute(0, 2, 3, 1).numpy().astype(np.int64)
        assert np.array_equal(y, synth.pack_codes(ref, bits))


@pytest.mark.parametrize("bits", [8, 4, 2, 1])
def test_linear_matches_matmul(orc, bits):
    rng = np.random.default_rng(70 + bits)
    k, n, m = 1024, 9, 10
    if bits == 1:
        xv = 2 * rng.integers(0, 2, size=(n, k)) - 1
        wv = 2 * rng.integers(0, 2, size=(m, k)) - 1
    else:
        xv = rng.integers(0, 1 << bits, size=(n, k))
        wv = rng.integers(-(1 << (bits - 1)), 1 << (bits - 1), size=(m, k))
    bias = rng.integers(-5000, 5000, size=m).astype(np.int32)
    acc, y = orc.linear(synth.pack_codes(synth.to_code(xv, bits, False), bits), n, k, bits,
                        synth.pack_codes(synth.to_code(wv, bits, True), bits), m, epi=2,
                        bias=bias, want_acc=True)
    ref = (torch.tensor(xv, dtype=torch.float64) @ torch.tensor(wv, dtype=torch.float64).T)
    ref = ref.numpy().astype(np.int64)
    assert np.array_equal(acc, ref)
    assert np.array_equal(y.astype(np.int64), ref + bias[None, :])


def test_relu_s8(orc):
    x = np.arange(-128, 128, dtype=np.int8)
    assert np.array_equal(orc.relu_s8(x), np.maximum(x, 0))


# ------------------------------------------------------- P11 shapes, MACs

def test_output_shape_formula(orc):
    for h in range(1, 12):
        for k in (1, 2, 3, 5):
            for s in (1, 2, 3):
                for p in (0, 1, 2):
                    if h + 2 * p < k:
                        assert orc.out_dim(h, k, s, p) == 0
                        continue
                    ref = F.conv2d(torch.zeros(1, 1, h, h, dtype=torch.float64),
                                   torch.zeros(1, 1, k, k, dtype=torch.float64),
                                   stride=s, padding=p).shape[-1]
                    assert orc.out_dim(h, k, s, p) == ref


def test_workload_mac_counts():
    assert synth.int8_layer().macs == 2_359_296
    assert synth.int4_layer().macs == 2_415_919_104
    assert synth.int2_layer().macs == 9_663_676_416
    assert synth.int1_layer().macs == 38_654_705_664
    net = synth.cifar_network(8, n=4096)
    assert synth.network_macs(net) == 12_298_240 * 4096 == 50_373_591_040
