#!/usr/bin/env python3
"""Throughput of the quantized convolution layer on one MI355X.

Metric: GMAC/s of one quantized conv layer at batch, and its fraction of the
dense int8 matrix-core peak.  The headline workload is the INT-4 3x3 layer on
a 64 x 32x32x64 batch with 64 filters; one "step" is one pass of the whole
layer (one launch of the fused conv + requantize + pack kernel) over the
batch.  Inputs sit in device memory (HBM) when the timed region starts.
Steps are captured in a HIP graph and replayed; the timed region is
bracketed by HIP events recorded on the stream the kernels run on.  Two
protocols, both reported for every workload:
  * warm: back-to-back launches on one resident input (a few MB, which the
    256 MB memory-side cache holds, as it holds a layer's input that the
    previous layer has just written);
  * cold: every timed step reads its own copy of the input and writes its
    own output buffer, and a 1 GiB device copy runs just before the timed
    region, so no step finds its data in the L2 or the memory-side cache.
The single layers (matrix-core or latency bound) are quoted warm, the
networks and their layers (whose first layers and classifier stream from
HBM) cold; "us_per_step" is the quoted one, "protocol" names it.

The other workloads (INT-8 batch 1, INT-2 batch 256 on the int8 and on the
FP4 matrix path, INT-1 batch 1024 on the XNOR and on the FP4 matrix path, the
INT-4 layer with the staircase epilogue, the CIFAR-shaped network at INT-8
and INT-4, batch 4096, whole and layer by layer) are reported under
"layers".  Measured denominators (int8 matrix-core loop, XNOR/popcount loop,
device copy, shader clock, empty launch) are taken in the same run
("calibration"), and the CPU oracle is timed on the host on every workload
("cpu_baseline").
"""
import argparse
import ctypes
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_INT8_TOPS = 5000.0        # MI355X dense int8 matrix-core peak, 10^12 int ops/s
PEAK_FP4_TFLOPS = 10100.0      # MI355X dense FP4 (e2m1) matrix-core peak, 10^12 flop/s
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E, GB/s
SPEC_CUS, SPEC_GHZ = 256, 2.4
VALU_LANE_OPS = SPEC_CUS * 64 * SPEC_GHZ * 1e9   # 32-bit vector lane-ops/s
XNOR_PEAK_BMACS = VALU_LANE_OPS * 16             # 2 lane-ops (xor, bcnt) per 32 binary MACs
PROFILES = os.path.join(ROOT, "profiles")
TRAFFIC = os.path.join(PROFILES, "conv_int4_32x32x64_m64_b64_traffic.txt")
COUNTERS = os.path.join(PROFILES, "conv_int4_32x32x64_m64_b64_counters.txt")
TRACE = os.path.join(PROFILES, "conv_int4_32x32x64_m64_b64_kernel_trace.md")
FLUSH_BYTES = 1 << 30          # evicts the 256 MB memory-side cache and every L2
COPIES_MAX_BYTES = 16 << 30    # device memory given to rotated input/output copies


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_sha():
    csrc = os.path.join(ROOT, "paper_1908_11263_amd", "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h")):
            with open(os.path.join(csrc, f), "rb") as fh:
                h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def read_summary(path):
    """The '@key: value' lines of a committed profile summary."""
    vals = {}
    if not os.path.exists(path):
        return vals
    with open(path) as f:
        for line in f:
            if line.startswith("@") and ":" in line:
                k, v = line[1:].split(":", 1)
                vals[k.strip()] = v.strip()
    return vals


def recorded_profile():
    """Evidence for the headline kernel from the committed rocprofv3
    summaries, each only if taken on the current kernel sources: the kernel
    name and average duration (kernel trace), HBM bytes per launch (PMC
    FETCH_SIZE / WRITE_SIZE), the SQ counters per launch."""
    sha = kernel_source_sha()
    out = {"kernel": None, "profile_avg_us": None, "traffic": None, "counters": None,
           "profiles_current": True}
    tr = read_summary(TRACE)
    if tr.get("kernel_source_sha") == sha:
        out["kernel"] = tr.get("headline_kernel")
        try:
            out["profile_avg_us"] = float(tr["headline_avg_us"])
        except (KeyError, ValueError):
            pass
    elif tr:
        out["profiles_current"] = False
    tf = read_summary(TRAFFIC)
    if tf.get("kernel_source_sha") == sha:
        try:
            out["traffic"] = int(tf["traffic_bytes_per_launch"])
        except (KeyError, ValueError):
            pass
    elif tf:
        out["profiles_current"] = False
    cn = read_summary(COUNTERS)
    if cn.get("kernel_source_sha") == sha:
        out["counters"] = {k: float(v) for k, v in cn.items()
                           if k not in ("kernel_source_sha", "kernel")}
    elif cn:
        out["profiles_current"] = False
    return out


# ----------------------------------------------------------------- steps

def _copies(footprint, steps):
    """Number of rotated input/output copies: one per timed step, within
    COPIES_MAX_BYTES (then at least 512 MB of data between reuses)."""
    return int(max(1, min(steps, COPIES_MAX_BYTES // max(1, footprint))))


class ConvStep:
    """One conv layer: `copies` device-resident copies of the input and as
    many output buffers; launch(i) runs qnn_conv2d (or qnn_conv2d_tiled) on
    copy i through ctypes with prebuilt descriptors."""

    def __init__(self, L, epi=None, tile=None, copies=1):
        import torch
        import paper_1908_11263_amd as qnn
        self.L = L
        epi = epi or L.epi
        q = qnn.qnn
        self.lib = q.lib()

        def d(a):
            return None if a is None else torch.from_numpy(a.copy()).cuda()
        x = d(L.x)
        w, b, mu, sh, th = (d(a) for a in (L.wt, L.bias, L.mult, L.shift, L.thresh))
        yshape = q.out_shape((L.n, L.h, L.w, L.c), L.bits, L.m, L.kh, L.kw, L.stride, L.pad, epi)
        y0 = q._out_tensor(yshape, None, x.device)
        self.copies = copies
        self.xs = x.unsqueeze(0).repeat(copies, *([1] * x.dim())).contiguous()
        self.ys = torch.empty((copies,) + tuple(y0.shape), dtype=y0.dtype, device=x.device)
        self.y = self.ys[0]
        del x, y0
        e, _ = q._epi(epi, b, mu, sh, th, L.clip)
        self._keep = (w, b, mu, sh, th, e)
        xd = q.Tensor(L.n, L.h, L.w, L.c, L.bits)
        yd = q.Tensor(*yshape)
        g = q.ConvGeom(L.kh, L.kw, L.stride[0], L.stride[1], L.pad[0], L.pad[1])
        self._desc = (xd, yd, g)
        self.tile = q.Tile(*tile) if tile is not None else None
        self.fn = self.lib.qnn_conv2d_tiled if tile is not None else self.lib.qnn_conv2d
        self.args = []
        for i in range(copies):
            a = [ctypes.byref(xd), ctypes.c_void_p(self.xs[i].data_ptr()), L.m,
                 ctypes.c_void_p(w.data_ptr()), ctypes.byref(g), ctypes.byref(e), ctypes.byref(yd),
                 ctypes.c_void_p(self.ys[i].data_ptr())]
            if tile is not None:
                a.insert(6, ctypes.byref(self.tile))
            self.args.append(a)
        self.macs = L.macs
        self.bytes = L.x.nbytes + L.wt.nbytes + self.y.numel() * self.y.element_size() + \
            sum(a.nbytes for a in (L.bias, L.mult, L.shift, L.thresh) if a is not None)
        self.footprint = L.x.nbytes + self.y.numel() * self.y.element_size()
        self.sha = L.digest()

    def launch(self, i=0):
        import torch
        st = self.fn(*self.args[i % self.copies], ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        if st != 0:
            raise RuntimeError("%s failed with status %d" % (self.fn.__name__, st))

    def try_launch(self):
        """One launch on the current stream; the status code (0 = launched)."""
        import torch
        return self.fn(*self.args[0], ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))


def _net_params(net, dev):
    import synth
    convs = []
    for cv in net.convs:
        wt = synth.pack_codes(synth.to_code(cv["w_vals"], net.bits, True).reshape(cv["m"], -1), net.bits)
        convs.append(dict(w=dev(wt), bias=dev(cv["bias"]), mult=dev(cv["mult"]), shift=dev(cv["shift"]),
                          m=cv["m"], k=5, pad=2, c=cv["c"], c_alg=cv["c_alg"], wbytes=wt.nbytes))
    fcw = synth.pack_codes(synth.to_code(net.fc_w_vals, net.bits, True), net.bits)
    fc = dict(w=dev(fcw), bias=dev(net.fc_bias), m=10, wbytes=fcw.nbytes)
    return convs, fc


class NetworkStep:
    """The CIFAR-shaped network (3 x conv + pool, FC) as one step, the input
    rotated over `copies` device copies."""

    def __init__(self, net, copies=1):
        import torch
        import synth
        self.net = net

        def d(a):
            return torch.from_numpy(a.copy()).cuda()
        self.convs, self.fc = _net_params(net, d)
        x = d(net.packed_input())
        self.copies = copies
        self.xs = x.unsqueeze(0).repeat(copies, 1, 1, 1, 1).contiguous()
        self.cin = net.x_vals.shape[-1]
        self.macs = synth.network_macs(net)
        self.bytes = None
        self.footprint = x.numel()
        self.sha = synth.sha256(net.packed_input(), *[cv["w_vals"] for cv in net.convs], net.fc_w_vals)

    def launch(self, i=0):
        from paper_1908_11263_amd.network import cifar_forward
        self.out = cifar_forward(self.xs[i % self.copies], self.net.n, self.net.bits, self.cin, self.convs,
                                 self.fc, self.net.clip)


class NetLayerStep:
    """One layer of the CIFAR-shaped network (a fused conv + pool, or the
    classifier) on the activations the network feeds it, rotated over
    `copies` input copies and output buffers."""

    def __init__(self, net, index, copies=1):
        import torch
        import paper_1908_11263_amd as qnn
        from paper_1908_11263_amd.network import cifar_forward
        self.q = qnn

        def d(a):
            return torch.from_numpy(a.copy()).cuda()
        convs, fc = _net_params(net, d)
        x = d(net.packed_input())
        cin = net.x_vals.shape[-1]
        _, acts = cifar_forward(x, net.n, net.bits, cin, convs, fc, net.clip, keep=True)
        torch.cuda.synchronize()
        inputs = [x] + acts
        self.net, self.index, self.bits = net, index, net.bits
        xin = inputs[index]
        hw = 32 >> index
        self.copies = copies
        self.xs = xin.unsqueeze(0).repeat(copies, *([1] * xin.dim())).contiguous()
        n = net.n
        if index < 3:
            cv = convs[index]
            self.layer = cv
            self.xshape = (n, hw, hw, cv["c"])
            self.ys = torch.empty((copies, n, hw // 2, hw // 2, cv["m"] * net.bits // 8), dtype=torch.uint8,
                                  device=x.device)
            self.macs = n * hw * hw * cv["m"] * 25 * cv["c_alg"]
            params = cv["m"] * 9
            self.name = "conv%d_pool" % (index + 1)
        else:
            self.layer = fc
            self.xshape = (n, hw, hw, convs[2]["m"])
            self.ys = torch.empty((copies, n, 1, 1, 10), dtype=torch.int32, device=x.device)
            self.macs = n * net.fc_w_vals.size
            params = 10 * 4
            self.name = "fc"
        self.bytes = xin.numel() + self.layer["wbytes"] + params + self.ys[0].numel() * self.ys.element_size()
        self.footprint = xin.numel() + self.ys[0].numel() * self.ys.element_size()
        del inputs, acts, x

    def launch(self, i=0):
        j = i % self.copies
        cv, q = self.layer, self.q
        if self.index < 3:
            q.conv2d_maxpool(self.xs[j], self.xshape, self.bits, cv["w"], cv["m"], 5, 5, (1, 1), (2, 2),
                             "requant", bias=cv["bias"], mult=cv["mult"], shift=cv["shift"], clip=self.net.clip,
                             out=self.ys[j])
        else:
            q.linear(self.xs[j], self.xshape, self.bits, cv["w"], 10, "raw32", bias=cv["bias"], out=self.ys[j])


class Flush:
    """A FLUSH_BYTES device copy (the library's measurement copy kernel)
    between two scratch buffers: afterwards no earlier data is cached."""

    def __init__(self):
        import torch
        self.a = torch.ones(FLUSH_BYTES, dtype=torch.uint8, device="cuda")
        self.b = torch.empty_like(self.a)

    def __call__(self):
        import torch
        st = calib_lib().qnn_calib_copy(ctypes.c_void_p(self.a.data_ptr()), ctypes.c_void_p(self.b.data_ptr()),
                                        FLUSH_BYTES, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        if st != 0:
            raise RuntimeError("qnn_calib_copy failed with status %d" % st)


def time_steps(step, steps, warmup, flush=None, graph=True):
    """Seconds per step.  Warm up, capture `steps` launches (launch i on copy
    i of the step's rotation) in one HIP graph, replay it once (upload), run
    the flush if given, then time one replay with events on the capture
    stream."""
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for i in range(warmup):
            step.launch(i)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    if graph:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for i in range(steps):
                step.launch(i)
        with torch.cuda.stream(s):
            g.replay()  # the first replay uploads the graph
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            if flush:
                flush()
            t0.record(s)
            g.replay()
            t1.record(s)
        torch.cuda.synchronize()
        del g
        return t0.elapsed_time(t1) / 1e3 / steps
    with torch.cuda.stream(s):
        if flush:
            flush()
        t0.record(s)
        for i in range(steps):
            step.launch(i)
        t1.record(s)
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / 1e3 / steps


# ----------------------------------------------------------- calibration

_calib = None


def calib_lib():
    global _calib
    if _calib is None:
        import paper_1908_11263_amd as qnn
        L = qnn.qnn.lib()
        P, i32 = ctypes.c_void_p, ctypes.c_int32
        for name in ("qnn_calib_mfma_i8", "qnn_calib_xnor"):
            f = getattr(L, name)
            f.restype = ctypes.c_int
            f.argtypes = [i32, i32, P, P, P]
        L.qnn_calib_copy.restype = ctypes.c_int
        L.qnn_calib_copy.argtypes = [P, P, ctypes.c_size_t, P]
        L.qnn_calib_empty.restype = ctypes.c_int
        L.qnn_calib_empty.argtypes = [i32, P]
        _calib = L
    return _calib


def _event_time(fn, reps=3):
    """Best wall time of fn() on the current stream over `reps` runs (HIP
    events around each run)."""
    import torch
    best = None
    for _ in range(reps):
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        fn()
        t1.record()
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1)
        best = ms if best is None else min(best, ms)
    return best / 1e3


def calibrate():
    """Measured denominators on this device: the int8 matrix-core rate, the
    XNOR/popcount rate, the copy bandwidth, the shader clock over each loop
    (shader-clock cycles per 100 MHz reference tick) and the empty launch."""
    import torch
    L = calib_lib()
    cus = torch.cuda.get_device_properties(0).multi_processor_count

    def stream():
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)

    def check(st, what):
        if st != 0:
            raise RuntimeError("%s failed with status %d" % (what, st))

    out = {"cus": cus}
    # int8 matrix cores: two workgroups (8 waves) per CU, 4 chains per wave
    blocks, iters = 2 * cus, 20000
    buf = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")
    clk = torch.zeros(2 * blocks, dtype=torch.int64, device="cuda")
    run = lambda: check(L.qnn_calib_mfma_i8(blocks, iters, ctypes.c_void_p(buf.data_ptr()),  # noqa: E731
                                            ctypes.c_void_p(clk.data_ptr()), stream()), "qnn_calib_mfma_i8")
    run()
    torch.cuda.synchronize()
    sec = _event_time(run)
    macs = blocks * 4 * iters * 4 * 32768
    c = clk.view(-1, 2).double().sum(0).tolist()
    out["mfma_i8"] = {"macs": macs, "seconds": round(sec, 6), "tops": round(2 * macs / sec / 1e12, 1),
                      "pct_of_spec": round(100 * 2 * macs / sec / 1e12 / PEAK_INT8_TOPS, 2),
                      "sclk_ghz": round(0.1 * c[0] / c[1], 3) if c[1] > 0 else None}
    # XNOR + popcount: eight workgroups (32 waves) per CU
    blocks, iters = 8 * cus, 4000
    buf = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")
    clk = torch.zeros(2 * blocks, dtype=torch.int64, device="cuda")
    run = lambda: check(L.qnn_calib_xnor(blocks, iters, ctypes.c_void_p(buf.data_ptr()),  # noqa: E731
                                         ctypes.c_void_p(clk.data_ptr()), stream()), "qnn_calib_xnor")
    run()
    torch.cuda.synchronize()
    sec = _event_time(run)
    bmacs = blocks * 256 * iters * 8 * 32
    c = clk.view(-1, 2).double().sum(0).tolist()
    out["xnor"] = {"bmacs_per_s": round(bmacs / sec, 1),
                   "pct_of_spec": round(100 * bmacs / sec / XNOR_PEAK_BMACS, 2),
                   "sclk_ghz": round(0.1 * c[0] / c[1], 3) if c[1] > 0 else None}
    # device copy of 1 GiB (read 1 GiB, write 1 GiB)
    nbytes = 1 << 30
    a = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    run = lambda: check(L.qnn_calib_copy(ctypes.c_void_p(a.data_ptr()), ctypes.c_void_p(b.data_ptr()),  # noqa
                                         nbytes, stream()), "qnn_calib_copy")
    run()
    torch.cuda.synchronize()
    sec = _event_time(run)
    out["copy"] = {"bytes": nbytes, "gbs": round(2 * nbytes / sec / 1e9, 1),
                   "pct_of_spec": round(100 * 2 * nbytes / sec / 1e9 / PEAK_HBM_GBS, 2)}
    del a, b
    # empty launches of 512 workgroups, graph-replayed
    class Empty:
        def launch(self, i=0):
            check(L.qnn_calib_empty(512, stream()), "qnn_calib_empty")
    out["empty_launch_us"] = round(time_steps(Empty(), 200, 10) * 1e6, 3)
    torch.cuda.empty_cache()
    return out


# --------------------------------------------------------- tile sweep

# Tile shapes built into the library: (kernel, tile_m, tile_n, waves);
# kernel 4 is the INT-2 path on the e2m1 (FP4) matrix instruction, kernel 1
# the image kernel (whole images or row bands in local memory).
TILE_FP4, TILE_IMAGE = 4, 1


def built_tiles(bits):
    out = [(TILE_IMAGE, 0, 0, 0)]
    out += [(16, m, n, 4) for m in (1, 2, 4) for n in (1, 2, 4)]
    out += [(32, m, n, w) for m in (1, 2) for n in (1, 2) for w in (4, 8)]
    if bits == 8:
        out.append((32, 4, 1, 4))
    if bits == 2:
        out.append((TILE_FP4, 0, 0, 0))
        out += [(TILE_FP4, m, n, w) for m in (1, 2) for n in (1, 2) for w in (4, 8)]
    return out


def tile_model(bits, tile):
    """Per wave and per K step of the tile: MACs, bytes read from LDS into
    registers (filter fragments, im2col fragments, the tap-offset table) and
    VALU ops spent expanding packed filter fragments, from the kernels'
    main loops.  16x16x64 kernel: every fragment is 64 lanes x 16 int8
    bytes, one 4-byte table entry per lane per step, weights staged unpacked.
    32x32x32 kernel: filter fragments stay packed (16*bits/8 bytes per lane)
    and are expanded in registers (INT-4: 3 ops per packed word, two words;
    INT-2: 7 ops per word), im2col fragments are 16 bytes per lane, one
    8-byte table entry per lane per pair of steps.  FP4 kernel (32x32x64
    e2m1): 16 bytes of nibbles per lane for each operand, no expansion.
    Image kernel: filter fragments in registers for the whole kernel, two
    32x32 row tiles per wave, 16 bytes of im2col per lane and tile.  (The
    library's own FP4 pick, tile_m = 0, has no fixed shape.)"""
    kern, tm, tn, _ = tile
    if kern == TILE_IMAGE:
        return {"macs_per_wave_kstep": 2 * 32 * 32 * 32, "lds_bytes_per_kmac": round(1024.0 * 64 * 32 / 65536, 1),
                "unpack_valu_per_mfma": 0.0, "acc_regs": 32}
    if tm == 0:
        return {}
    if kern == TILE_FP4:
        macs = tm * tn * 32 * 32 * 64
        lds = 64 * 16 * (tm + tn) + 64 * 4
        valu = 0
    elif kern == 16:
        macs = tm * tn * 16 * 16 * 64
        lds = 64 * 16 * (tm + tn) + 64 * 4
        valu = 0
    else:
        macs = tm * tn * 32 * 32 * 32
        lds = 64 * (2 * bits) * tm + 64 * 16 * tn + 64 * 4
        valu = tm * {8: 0, 4: 6, 2: 7}[bits]
    return {"macs_per_wave_kstep": macs, "lds_bytes_per_kmac": round(1024.0 * lds / macs, 1),
            "unpack_valu_per_mfma": round(valu / float(tm * tn), 2),
            "acc_regs": tm * tn * (4 if kern == 16 else 16)}


def tile_sweep(args):
    """Every built tile shape on the INT-8/4/2 3x3 32x32x64 batch-64 layers
    and the INT-2 16x16x128 batch-256 layer: one JSON line per (layer, tile)
    with its time per step (graph replay, warm caches), throughput, the
    analytic per-step model and whether the output equals the library's own
    choice bit for bit; refused shapes carry the status code instead."""
    import torch
    import synth
    layers = [synth.headline_shape_layer(8), synth.int4_layer(), synth.headline_shape_layer(2),
              synth.int2_layer()]
    for L in layers:
        auto = ConvStep(L)
        graph = not args.no_graph
        sec = time_steps(auto, args.steps, args.warmup, graph=graph)
        torch.cuda.synchronize()
        ref = auto.y.clone()
        rows = [dict(layer=L.name, tile="auto", us=round(sec * 1e6, 3),
                     gmacs=round(L.macs / sec / 1e9, 1),
                     pct_int8_mfma_peak=round(100 * 2 * L.macs / sec / 1e12 / PEAK_INT8_TOPS, 2))]
        for t in built_tiles(L.bits):
            step = ConvStep(L, tile=t)
            step.y.fill_(0)
            st = step.try_launch()
            torch.cuda.synchronize()
            row = dict(layer=L.name, tile=list(t), **tile_model(L.bits, t))
            if st != 0:
                row["status"] = st
            else:
                row["equal_to_auto"] = bool(torch.equal(step.y, ref))
                sec = time_steps(step, args.steps, args.warmup, graph=graph)
                row.update(us=round(sec * 1e6, 3), gmacs=round(L.macs / sec / 1e9, 1),
                           pct_int8_mfma_peak=round(100 * 2 * L.macs / sec / 1e12 / PEAK_INT8_TOPS, 2))
            rows.append(row)
            log("  %s tile %s: %s" % (L.name, t, "status %d" % st if st else "%.3f us" % row["us"]))
            del step
        for r in rows:
            print(json.dumps(r), flush=True)
        del auto
        torch.cuda.empty_cache()


# --------------------------------------------------------- CPU baseline

def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or None


def oracle_network(orc, net, images, threads):
    """Logits of the network on the oracle for the given images (conv, then
    max-pooling, per layer; then the classifier)."""
    import synth
    x = net.packed_input()[images]
    n = x.shape[0]
    h, c = 32, x.shape[-1] * 8 // net.bits
    for cv in net.convs:
        wt = synth.pack_codes(synth.to_code(cv["w_vals"], net.bits, True).reshape(cv["m"], -1), net.bits)
        _, y = orc.conv2d(x, (n, h, h, c), net.bits, wt, cv["m"], 5, 5, (1, 1), (2, 2), orc.REQUANT,
                          cv["bias"], cv["mult"], cv["shift"], None, net.clip, nthreads=threads)
        c = cv["m"]
        x = orc.maxpool2d(y, (n, h, h, c), net.bits, 2, 2, 2, 2)
        h //= 2
    fcw = synth.pack_codes(synth.to_code(net.fc_w_vals, net.bits, True), net.bits)
    _, logits = orc.linear(x, n, h * h * c, net.bits, fcw, 10, epi=orc.RAW32, bias=net.fc_bias)
    return logits


def cpu_baseline(min_seconds=10.0):
    """The oracle (unchanged) on the host cores: the INT-4 workload repeated
    for at least `min_seconds` (the reported value), then one timed sample of
    every other workload, and the INT-8 batch-1 layer on one thread."""
    import numpy as np
    import oracle
    import synth
    try:
        host_cores = len(os.sched_getaffinity(0))
    except AttributeError:
        host_cores = os.cpu_count() or 1
    # at most 16 threads: the host's CPU share for one GPU on a shared machine
    threads = max(1, min(16, host_cores))
    oracle.build()

    def conv(L, idx, nthreads):
        x = L.x if idx is None else L.x[idx]
        n = x.shape[0]
        oracle.conv2d(x, (n, L.h, L.w, L.c), L.bits, L.wt, L.m, L.kh, L.kw, L.stride, L.pad,
                      {"requant": oracle.REQUANT, "thresh1": oracle.THRESH1, "stair": oracle.STAIR}[L.epi],
                      L.bias, L.mult, L.shift, L.thresh, L.clip, nthreads=nthreads)

    per = {}

    def record(name, macs, sec, images, nthreads):
        per[name] = {"seconds": round(sec, 4), "images": images, "threads": nthreads,
                     "gmacs": round(macs / sec / 1e9, 4)}

    L = synth.int4_layer()
    reps, t0 = 0, time.perf_counter()
    while True:
        conv(L, None, threads)
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_seconds:
            break
    record("int4", L.macs * reps, el, L.n * reps, threads)
    head = per["int4"]
    L8 = synth.int8_layer()
    for nthreads, key in ((1, "int8_1thread"), (threads, "int8")):
        reps, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < 1.0:
            conv(L8, None, nthreads)
            reps += 1
        record(key, L8.macs * reps, time.perf_counter() - t0, reps, nthreads)
    for name, mk, k in (("int2", synth.int2_layer, 32), ("int1", synth.int1_layer, 128),
                        ("int4_stair", synth.int4_stair_layer, 64)):
        Lx = mk()
        idx = np.arange(k)
        t0 = time.perf_counter()
        conv(Lx, idx, threads)
        record(name, Lx.macs * k // Lx.n, time.perf_counter() - t0, k, threads)
    for bits in (8, 4):
        net = synth.cifar_network(bits, n=4096)
        k = 64
        t0 = time.perf_counter()
        oracle_network(oracle, net, np.arange(k), threads)
        record("cifar%d" % bits, synth.network_macs(net) * k // net.n, time.perf_counter() - t0, k, threads)
    return {"value": head["gmacs"], "unit": "GMAC/s", "cores": threads, "kind": "oracle",
            "sample": "whole 64-image INT-4 batch x %d repetitions (%.1f s wall on %d threads); "
                      "per_config: one sample of each other workload" % (head["images"] // 64, head["seconds"],
                                                                          threads),
            "host_cores": host_cores, "cpu_model": cpu_model(), "per_config": per}


# ----------------------------------------------------------------- main

def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--only", default=None,
                    help="run only this workload (int8, int4, int2, int2_fp4, int1, int1_fp4, int4_stair, "
                         "cifar8, cifar4, cifar8_layers, cifar4_layers)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-calib", action="store_true", help="skip the measured denominators")
    ap.add_argument("--primary-only", action="store_true",
                    help="time each workload under its quoted protocol only (warm single layers, cold networks)")
    ap.add_argument("--no-graph", action="store_true", help="launch every step from Python")
    ap.add_argument("--tile-sweep", action="store_true",
                    help="time every built tile shape instead (one JSON line per layer and tile)")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="also run one device copy of this many bytes (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build measures the single-GPU path only; "
              "--gpus %d is not supported (run with --gpus 1)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import synth
    import paper_1908_11263_amd as qnn
    torch.cuda.set_device(0)
    qnn.device_check()
    graph = not args.no_graph

    if args.copy_bytes:
        nbytes = args.copy_bytes // 16 * 16
        a = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        st = calib_lib().qnn_calib_copy(ctypes.c_void_p(a.data_ptr()), ctypes.c_void_p(b.data_ptr()), nbytes,
                                        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        torch.cuda.synchronize()
        log("copy calibration: %d bytes, status %d" % (nbytes, st))
        del a, b

    if args.tile_sweep:
        tile_sweep(args)
        return

    calib = None if (args.no_calib or args.only) else calibrate()
    if calib:
        log("calibration:", json.dumps(calib))
    flush = Flush()

    workloads = {
        "int8": lambda c: ConvStep(synth.int8_layer(), copies=c),
        "int4": lambda c: ConvStep(synth.int4_layer(), copies=c),
        "int2": lambda c: ConvStep(synth.int2_layer(), copies=c),
        "int2_fp4": lambda c: ConvStep(synth.int2_layer(), tile=(TILE_FP4, 0, 0, 0), copies=c),
        "int1": lambda c: ConvStep(synth.int1_layer(), copies=c),
        "int1_fp4": lambda c: ConvStep(synth.int1_layer(), tile=(TILE_FP4, 0, 0, 0), copies=c),
        "int4_stair": lambda c: ConvStep(synth.int4_stair_layer(), copies=c),
        "cifar8": lambda c: NetworkStep(synth.cifar_network(8, n=4096), copies=c),
        "cifar4": lambda c: NetworkStep(synth.cifar_network(4, n=4096), copies=c),
    }
    footprints = {"int8": 8192 * 2, "int4": 4 << 20, "int2": 4 << 20, "int2_fp4": 4 << 20, "int1": 4 << 20,
                  "int1_fp4": 4 << 20, "int4_stair": 4 << 20, "cifar8": 16 << 20, "cifar4": 16 << 20}
    head = "int4"
    extra = ["cifar8_layers", "cifar4_layers"]
    names = [args.only] if args.only else [head] + [k for k in workloads if k != head] + extra

    layers = {}
    for name in names:
        steps = args.steps if name == head else max(20, min(args.steps, 200 if "cifar" in name else args.steps))
        warm = args.warmup if name == head else min(args.warmup, 10)
        if name in extra:
            bits = 8 if name == "cifar8_layers" else 4
            net = synth.cifar_network(bits, n=4096)
            rec = {}
            for i in range(4):
                probe = NetLayerStep(net, i, copies=1)
                copies = _copies(probe.footprint, steps)
                del probe
                step = NetLayerStep(net, i, copies=copies)
                sec = time_steps(step, steps, warm, flush=flush, graph=graph)
                r = {"macs_per_step": step.macs, "us_per_step": round(sec * 1e6, 3),
                     "gmacs": round(step.macs / sec / 1e9, 2),
                     "pct_int8_mfma_peak": round(100 * 2 * step.macs / sec / 1e12 / PEAK_INT8_TOPS, 3),
                     "algorithmic_bytes": step.bytes, "algorithmic_gbs": round(step.bytes / sec / 1e9, 1),
                     "pct_hbm_peak": round(100 * step.bytes / sec / 1e9 / PEAK_HBM_GBS, 2),
                     "copies": copies}
                rec[step.name] = r
                log("  %s %s: %.3f us/step, %.1f GMAC/s, %.1f GB/s" % (name, step.name, sec * 1e6,
                                                                       r["gmacs"], r["algorithmic_gbs"]))
                del step
                torch.cuda.empty_cache()
            layers[name] = rec
            continue
        cold_primary = "cifar" in name
        need_cold = cold_primary or not args.primary_only
        copies = _copies(footprints[name], steps) if need_cold else 1
        step = workloads[name](copies)
        log("workload %s: warmup %d, steps %d, %d input copies" % (name, warm, steps, copies))
        sw = sc = None
        if not cold_primary or not args.primary_only:
            step.copies = 1
            sw = time_steps(step, steps, warm, graph=graph)
            step.copies = copies
        if need_cold:
            sc = time_steps(step, steps, warm, flush=flush, graph=graph)
        sec = sc if cold_primary else sw
        gmacs = step.macs / sec / 1e9
        rec = {"macs_per_step": step.macs, "us_per_step": round(sec * 1e6, 3),
               "protocol": "cold" if cold_primary else "warm", "steps": steps,
               "gmacs": round(gmacs, 2),
               "pct_int8_mfma_peak": round(100 * 2 * step.macs / sec / 1e12 / PEAK_INT8_TOPS, 3),
               "copies": copies, "input_sha256": step.sha}
        if sw is not None:
            rec["us_per_step_warm"] = round(sw * 1e6, 3)
        if sc is not None:
            rec["us_per_step_cold"] = round(sc * 1e6, 3)
        if name in ("int2_fp4", "int1_fp4"):
            rec["pct_fp4_mfma_peak"] = round(100 * 2 * step.macs / sec / 1e12 / PEAK_FP4_TFLOPS, 3)
        if name == "int1":
            rec["pct_xnor_valu_roofline"] = round(100 * step.macs / sec / XNOR_PEAK_BMACS, 3)
            if calib:
                rec["pct_xnor_measured"] = round(100 * step.macs / sec / calib["xnor"]["bmacs_per_s"], 2)
        if name == "int8" and calib:
            rec["empty_launch_us"] = calib["empty_launch_us"]
        if "cifar" in name:
            rec["images_per_s"] = round(step.net.n / sec, 1)
        if step.bytes:
            rec["algorithmic_gbs"] = round(step.bytes / sec / 1e9, 2)
        if calib and name not in ("int1", "int1_fp4", "int2_fp4"):
            rec["pct_int8_mfma_measured"] = round(100 * 2 * step.macs / sec / 1e12 / calib["mfma_i8"]["tops"], 3)
        layers[name] = rec
        log("  %s: %.3f us/step %s (warm %s, cold %s), %.1f GMAC/s, %.2f%% of int8 MFMA peak"
            % (name, sec * 1e6, rec["protocol"], rec.get("us_per_step_warm"), rec.get("us_per_step_cold"),
               gmacs, rec["pct_int8_mfma_peak"]))
        if name == head:
            head_step, head_sec, head_done = step, sec, steps
        else:
            del step
            torch.cuda.empty_cache()

    if head not in layers:
        if args.only:
            print(json.dumps({"only": args.only, "layers": layers}), flush=True)
        return
    L = head_step.L
    ops = 2 * head_step.macs
    achieved = ops / head_sec / 1e12
    prof = recorded_profile()
    roofline = {"bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_INT8_TOPS,
                "unit": "TOP/s", "frac": round(achieved / PEAK_INT8_TOPS, 5),
                "traffic": prof["traffic"], "kernel": prof["kernel"], "ops_per_launch": ops,
                "algorithmic_bytes_per_launch": head_step.bytes}
    if prof["profile_avg_us"]:
        roofline["profile_avg_us"] = prof["profile_avg_us"]
        roofline["profile_frac"] = round(ops / (prof["profile_avg_us"] * 1e-6) / 1e12 / PEAK_INT8_TOPS, 5)
    if prof["counters"]:
        roofline["counters"] = prof["counters"]
    if not prof["profiles_current"]:
        roofline["profiles_note"] = "committed profile summaries predate the current kernel sources"
    if calib:
        roofline["measured_peak"] = calib["mfma_i8"]["tops"]
        roofline["frac_of_measured_peak"] = round(achieved / calib["mfma_i8"]["tops"], 5)
    hc = layers[head].get("us_per_step_cold")
    if hc:
        roofline["cold"] = {"us_per_step": hc, "achieved": round(ops / (hc * 1e-6) / 1e12, 3),
                            "frac": round(ops / (hc * 1e-6) / 1e12 / PEAK_INT8_TOPS, 5)}
    out = {
        "metric": "GMAC/s per qconv layer at INT8/4/2/1 (batch), % of int8 MFMA peak",
        "value": round(head_step.macs / head_sec / 1e9, 2),
        "unit": "GMAC/s",
        "n_gpus": 1, "steps": head_done, "warmup": args.warmup,
        "ms_per_step": round(head_sec * 1e3, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int8", "data": "synthetic",
        "config": {"workload": "int4_conv3x3_b64_32x32x64_m64", "bits": 4, "batch": L.n,
                   "h": L.h, "w": L.w, "c": L.c, "m": L.m, "kernel": 3, "stride": 1, "pad": 1,
                   "epilogue": "requant", "graph_replay": graph, "protocol": "warm"},
        "roofline": roofline,
        "layers": layers,
        "numpy": np.__version__,
    }
    if calib:
        out["calibration"] = calib
    if not args.no_cpu and not args.only:
        log("cpu baseline (oracle) ...")
        out["cpu_baseline"] = cpu_baseline()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
