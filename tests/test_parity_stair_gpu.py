"""GPU parity of the staircase epilogue (Sec. III-A, Eq. (4)): the HIP path
through the C ABI against the CPU oracle, byte for byte, on both conv
kernels (layers narrower than 32 channels or with few tiles run on the
16x16 kernel, the others on the 32x32 kernel)."""
import numpy as np
import pytest

import synth
from gpu_helpers import compare, gpu_conv, log, oracle_conv, with_epi

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def qnn():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1908_11263_amd as q
    q.device_check()
    return q


def check(orc, L):
    log("case", L.name, "stair N=%d H=%d W=%d C=%d M=%d k=%d bits=%d" % (
        L.n, L.h, L.w, L.c, L.m, L.kh, L.bits))
    got = gpu_conv(L)
    compare(got, oracle_conv(orc, L), L.name)
    return got


def stair_layer(bits, n, h, w, c, m, k, seed, sorted_=True, span=None):
    hi = (1 << bits) - 1
    whi = (1 << (bits - 1)) - 1
    span = span or max(1, k * k * c * hi * whi // 4)
    return synth.conv_layer("stair_int%d" % bits, bits, n, h, w, c, m, k, k // 2, seed, (0, hi),
                            (-(1 << (bits - 1)), whi), bias_rng=(-hi * 64, hi * 64),
                            thresh_rng=(-span, span), epi="stair", stair_sorted=sorted_)


def derived_thresholds(L):
    """Thresholds on acc + bias that reproduce L's multiplier/shift/clip
    compression (clip from 0 to 2^bits - 1)."""
    nt = (1 << L.bits) - 1
    tau = np.zeros((L.m, nt), dtype=np.int64)
    for j in range(L.m):
        s, M = int(L.shift[j]), int(L.mult[j])
        half = (1 << (s - 1)) if s else 0
        for p in range(1, nt + 1):
            tau[j, p - 1] = -((half - p * (1 << s)) // M)
    return tau


@pytest.mark.parametrize("bits", [4, 2])
def test_stair_random_small_layers(qnn, orc, bits):
    rng = np.random.default_rng(2000 + bits)
    for _ in range(16):
        check(orc, synth.random_small_layer(rng, bits, epi="stair"))


@pytest.mark.parametrize("bits", [4, 2])
def test_stair_both_kernels_ragged_channels(qnn, orc, bits):
    unit = 32 // bits
    for m in (5, 17, 33, 40, 70):
        # few tiles: the 16x16 kernel
        check(orc, stair_layer(bits, 2, 7, 9, 2 * unit, m, 3, seed=m))
        # enough tiles for the 32x32 kernel when m >= 32
        check(orc, stair_layer(bits, 24, 32, 32, 2 * unit, m, 3, seed=100 + m))


@pytest.mark.parametrize("bits", [4, 2])
def test_stair_unsorted_thresholds(qnn, orc, bits):
    unit = 32 // bits
    for (n, h, w, m) in ((2, 6, 5, 20), (24, 32, 32, 64)):
        L = stair_layer(bits, n, h, w, 2 * unit, m, 3, seed=7 * m, sorted_=False)
        assert (np.diff(L.thresh, axis=1) < 0).any()
        check(orc, L)


@pytest.mark.parametrize("which", ["int4", "int2"])
def test_stair_with_derived_thresholds_equals_requant(qnn, orc, which):
    """A workload layer (centred bias) run with the thresholds of its own
    multiplier/shift: the staircase output equals the requantized output, on
    the GPU, and the staircase output equals the oracle's."""
    L = synth.centred(synth.int4_layer() if which == "int4" else synth.int2_layer())
    hi = (1 << L.bits) - 1
    assert L.clip == (0, hi)
    tau = derived_thresholds(L)
    assert np.abs(tau).max() < 1 << 31
    S = with_epi(L, "stair")
    S.thresh = tau.astype(np.int32)
    got_req = gpu_conv(L)
    got = check(orc, S)
    assert np.array_equal(gpu_conv(S), got_req)
    del got


def test_stair_extreme_thresholds(qnn, orc):
    """Thresholds at the ends of int32 and a bias that moves them past it."""
    for bits in (4, 2):
        unit = 32 // bits
        for m in (8, 48):
            L = stair_layer(bits, 16 if m > 32 else 2, 16, 16, 2 * unit, m, 3, seed=m + bits)
            nt = (1 << bits) - 1
            t = L.thresh.astype(np.int64)
            t[:, 0] = -(1 << 31)
            t[:, -1] = (1 << 31) - 1
            L.thresh = np.sort(t, axis=1).astype(np.int32)
            L.bias = np.where(np.arange(m) % 2 == 0, (1 << 31) - 1, -(1 << 31)).astype(np.int32)
            check(orc, L)
            del nt


def test_stair_bench_workload(qnn, orc):
    """The benchmarked staircase layer (INT4, batch 64, 32x32x64 -> 64)."""
    L = synth.int4_stair_layer()
    y = check(orc, L)
    codes = np.concatenate([(y & 15).ravel(), (y >> 4).ravel()])
    log("int4 stair codes: min %d max %d distinct %d" % (codes.min(), codes.max(), len(np.unique(codes))))
