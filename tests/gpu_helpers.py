"""Shared helpers for the GPU parity tests: run a layer through the C ABI
(via the ctypes binding) and through the CPU oracle on the same seeded
inputs."""
import os
import sys

import numpy as np

import synth

EPI = {"requant": 0, "thresh1": 1, "raw32": 2, "stair": 3}


def threads():
    """Oracle threads: the host cores available, at most 16 (the CPU share
    that goes with one GPU on a shared GPU host; more threads there would
    take cores from other jobs' processes)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def dev(a):
    import torch
    if a is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def gpu_conv(L, epi=None, stream=None):
    """Run layer L on the GPU through qnn_conv2d; returns a numpy array."""
    import torch
    import paper_1908_11263_amd as qnn
    epi = epi or L.epi
    y = qnn.conv2d(dev(L.x), (L.n, L.h, L.w, L.c), L.bits, dev(L.wt), L.m, L.kh, L.kw, L.stride,
                   L.pad, epi, bias=dev(L.bias), mult=dev(L.mult), shift=dev(L.shift),
                   thresh=dev(L.thresh), clip=L.clip, stream=stream)
    torch.cuda.synchronize()
    return y.cpu().numpy()


# whole oracle outputs of the large workloads, kept for the session: the
# integer and the FP4 paths of a layer are both compared with one oracle run
_ORACLE_CACHE = {}


def oracle_conv(orc, L, epi=None):
    """Oracle output of layer L (the whole batch); outputs of layers of more
    than 2^28 MACs are cached per (input digest, epilogue)."""
    epi = epi or L.epi
    key = (L.name, L.digest(), epi)
    if key in _ORACLE_CACHE:
        return _ORACLE_CACHE[key]
    _, y = orc.conv2d(L.x, (L.n, L.h, L.w, L.c), L.bits, L.wt, L.m, L.kh, L.kw, L.stride, L.pad,
                      EPI[epi], L.bias, L.mult, L.shift, L.thresh, L.clip, nthreads=threads())
    if L.macs > (1 << 28):
        _ORACLE_CACHE[key] = y
    return y


def compare(got, want, what):
    """Byte-for-byte equality of two outputs, naming the first mismatches."""
    assert got.shape == want.shape, "%s: shape %s, oracle %s" % (what, got.shape, want.shape)
    bad = np.argwhere(got != want)
    assert bad.size == 0, "%s: %d mismatches of %d, first at %s" % (
        what, len(bad), got.size, bad[:5].tolist())


def with_epi(L, epi):
    """The same tensors with another epilogue (bias kept)."""
    out = synth.ConvLayer(L.name + "_" + epi, L.bits, L.n, L.h, L.w, L.c, L.m, L.kh, L.kw,
                          L.stride, L.pad, epi, L.x_vals, L.w_vals, L.bias, L.mult, L.shift,
                          L.thresh, L.clip, L.c_alg)
    return out


def distribution(y_codes, bits):
    """Fractions of output codes at 0, at the top code, and in between."""
    y = np.asarray(y_codes, dtype=np.uint8)
    fields = np.unpackbits(y[..., None], axis=-1, bitorder="little").reshape(-1, 8 // bits, bits)
    codes = (fields * (1 << np.arange(bits))).sum(axis=-1).ravel()
    hi = (1 << bits) - 1
    return float((codes == 0).mean()), float((codes == hi).mean())
