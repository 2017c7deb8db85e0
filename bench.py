#!/usr/bin/env python3
"""Throughput of the quantized convolution layer on one MI355X.

Metric: GMAC/s of one quantized conv layer at batch, and its fraction of the
dense int8 matrix-core peak.  The headline workload is the INT-4 3x3 layer on
a 64 x 32x32x64 batch with 64 filters; one "step" is one pass of the whole
layer (one launch of the fused conv + requantize + pack kernel) over the
batch, inputs resident in device memory.  Steps are captured in a HIP graph
and replayed; the timed region is bracketed by HIP events recorded on the
stream the kernels run on.  The other workloads (INT-8 batch 1, INT-2 batch
256 on the int8 and on the FP4 matrix path, INT-1 batch 1024 on the XNOR
and on the FP4 matrix path, the INT-4
layer with the staircase epilogue, the CIFAR-shaped network at INT-8 and
INT-4, batch 4096) are reported under "layers".  The CPU oracle is timed on the host on
the same INT-4 workload for the "cpu_baseline" object.
"""
import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_INT8_TOPS = 5000.0        # MI355X dense int8 matrix-core peak, 10^12 int ops/s
PEAK_FP4_TFLOPS = 10100.0      # MI355X dense FP4 (e2m1) matrix-core peak, 10^12 flop/s
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E, GB/s
VALU_LANE_OPS = 256 * 64 * 2.4e9   # 32-bit vector lane-ops/s: 256 CUs x 64 lanes x 2.4 GHz
XNOR_PEAK_BMACS = VALU_LANE_OPS * 16  # 2 lane-ops (xnor, bcnt) per 32 binary MACs
PROFILE = os.path.join(ROOT, "profiles", "conv_int4_32x32x64_m64_b64_traffic.txt")


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


def recorded_profile():
    """(HBM bytes per launch, kernel name) of the headline kernel from the
    committed PMC summary; the byte count only if the summary was taken on the
    current kernel sources."""
    if not os.path.exists(PROFILE):
        return None, None
    vals = {}
    name = None
    with open(PROFILE) as f:
        for line in f:
            if line.startswith("# HBM traffic of "):
                name = line[len("# HBM traffic of "):].split(" (")[0].strip()
            if ":" in line and line.startswith("@"):
                k, v = line[1:].split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_source_sha") != kernel_source_sha():
        return None, name
    try:
        return int(vals["traffic_bytes_per_launch"]), name
    except (KeyError, ValueError):
        return None, name


class ConvStep:
    """One conv layer with device-resident inputs and preallocated output;
    launch() calls qnn_conv2d through ctypes with prebuilt descriptors."""

    def __init__(self, L, epi=None, tile=None):
        import torch
        import paper_1908_11263_amd as qnn
        self.L = L
        epi = epi or L.epi
        q = qnn.qnn
        self.lib = q.lib()

        def d(a):
            return None if a is None else torch.from_numpy(a.copy()).cuda()
        self.keep = [d(L.x), d(L.wt), d(L.bias), d(L.mult), d(L.shift), d(L.thresh)]
        x, w, b, mu, sh, th = self.keep
        yshape = q.out_shape((L.n, L.h, L.w, L.c), L.bits, L.m, L.kh, L.kw, L.stride, L.pad, epi)
        self.y = q._out_tensor(yshape, None, x.device)
        e, _ = q._epi(epi, b, mu, sh, th, L.clip)
        self.args = [ctypes.byref(q.Tensor(L.n, L.h, L.w, L.c, L.bits)), ctypes.c_void_p(x.data_ptr()),
                     L.m, ctypes.c_void_p(w.data_ptr()),
                     ctypes.byref(q.ConvGeom(L.kh, L.kw, L.stride[0], L.stride[1], L.pad[0], L.pad[1])),
                     ctypes.byref(e), ctypes.byref(q.Tensor(*yshape)), ctypes.c_void_p(self.y.data_ptr())]
        if tile is not None:
            # qnn_conv2d_tiled takes the tile descriptor before the output
            self.tile = q.Tile(*tile)
            self.args.insert(6, ctypes.byref(self.tile))
        self.fn = self.lib.qnn_conv2d_tiled if tile is not None else self.lib.qnn_conv2d
        self._refs = (e,)
        self.macs = L.macs
        self.bytes = L.x.nbytes + L.wt.nbytes + self.y.numel() * self.y.element_size() + \
            sum(a.nbytes for a in (L.bias, L.mult, L.shift, L.thresh) if a is not None)

    def launch(self):
        import torch
        st = self.fn(*self.args, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        if st != 0:
            raise RuntimeError("%s failed with status %d" % (self.fn.__name__, st))

    def try_launch(self):
        """One launch on the current stream; the status code (0 = launched)."""
        import torch
        return self.fn(*self.args, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))


class NetworkStep:
    """The CIFAR-shaped network (3 conv + pool, FC) as one step."""

    def __init__(self, net):
        import torch
        import synth
        self.net = net

        def d(a):
            return torch.from_numpy(a.copy()).cuda()
        self.convs = []
        for cv in net.convs:
            wt = synth.pack_codes(synth.to_code(cv["w_vals"], net.bits, True).reshape(cv["m"], -1),
                                  net.bits)
            self.convs.append(dict(w=d(wt), bias=d(cv["bias"]), mult=d(cv["mult"]),
                                   shift=d(cv["shift"]), m=cv["m"], k=5, pad=2))
        self.fc = dict(w=d(synth.pack_codes(synth.to_code(net.fc_w_vals, net.bits, True), net.bits)),
                       bias=d(net.fc_bias), m=10)
        self.x = d(net.packed_input())
        self.cin = net.x_vals.shape[-1]
        self.macs = synth.network_macs(net)
        self.bytes = None

    def launch(self):
        from paper_1908_11263_amd.network import cifar_forward
        self.out = cifar_forward(self.x, self.net.n, self.net.bits, self.cin, self.convs, self.fc,
                                 self.net.clip)


def time_steps(step, steps, warmup, graph=True, per_graph=50):
    """Seconds per step: warm up, capture `per_graph` steps in a HIP graph,
    replay until `steps` steps ran, time with events on the capture stream."""
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for _ in range(warmup):
            step.launch()
    torch.cuda.synchronize()
    if graph:
        per_graph = max(1, min(per_graph, steps))
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            for _ in range(per_graph):
                step.launch()
        reps = max(1, steps // per_graph)
        done = reps * per_graph
        with torch.cuda.stream(s):
            g.replay()  # first replay uploads the graph
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            t0.record(s)
            for _ in range(reps):
                g.replay()
            t1.record(s)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / 1e3 / done, done
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        t0.record(s)
        for _ in range(steps):
            step.launch()
        t1.record(s)
    torch.cuda.synchronize()
    return t0.elapsed_time(t1) / 1e3 / steps, steps


# Tile shapes built into the library: (kernel, tile_m, tile_n, waves);
# kernel 4 is the INT-2 path on the e2m1 (FP4) matrix instruction.
TILE_FP4 = 4


def built_tiles(bits):
    out = [(16, m, n, 4) for m in (1, 2, 4) for n in (1, 2, 4)]
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
    (The FP4 library pick, tile_m = 0, has no fixed shape.)"""
    kern, tm, tn, _ = tile
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
    with its time per step (graph replay), throughput, the analytic per-step
    model and whether the output equals the library's own choice bit for
    bit; refused shapes carry the status code instead."""
    import torch
    import synth
    layers = [synth.headline_shape_layer(8), synth.int4_layer(), synth.headline_shape_layer(2),
              synth.int2_layer()]
    for L in layers:
        auto = ConvStep(L)
        graph = not args.no_graph
        sec, done = time_steps(auto, args.steps, args.warmup, graph=graph)
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
                sec, done = time_steps(step, args.steps, args.warmup, graph=graph)
                row.update(us=round(sec * 1e6, 3), gmacs=round(L.macs / sec / 1e9, 1),
                           pct_int8_mfma_peak=round(100 * 2 * L.macs / sec / 1e12 / PEAK_INT8_TOPS, 2))
            rows.append(row)
            log("  %s tile %s: %s" % (L.name, t, "status %d" % st if st else "%.3f us" % row["us"]))
            del step
        for r in rows:
            print(json.dumps(r), flush=True)
        del auto
        torch.cuda.empty_cache()


def cpu_baseline(L, min_seconds=10.0):
    """The oracle (unchanged) on the host cores over the same INT-4 workload,
    repeated until at least `min_seconds` of wall time."""
    import oracle
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    threads = max(1, min(16, cores))
    oracle.build()
    reps = 0
    t0 = time.perf_counter()
    while True:
        oracle.conv2d(L.x, (L.n, L.h, L.w, L.c), L.bits, L.wt, L.m, L.kh, L.kw, L.stride, L.pad,
                      oracle.REQUANT, L.bias, L.mult, L.shift, None, L.clip, nthreads=threads)
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_seconds:
            break
    return {"value": round(L.macs * reps / el / 1e9, 4), "unit": "GMAC/s", "cores": threads,
            "kind": "oracle",
            "sample": "whole %d-image INT-4 batch x %d repetitions (%.1f s wall on %d threads)"
                      % (L.n, reps, el, threads)}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--only", default=None,
                    help="run only this workload (int8, int4, int2, int2_fp4, int1, int1_fp4, int4_stair, cifar8, cifar4)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-graph", action="store_true", help="launch every step from Python")
    ap.add_argument("--tile-sweep", action="store_true",
                    help="time every built tile shape instead (one JSON line per layer and tile)")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="also run one plain device copy of this many bytes (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build measures the single-GPU path only; "
              "--gpus %d is not supported (run with --gpus 1)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    import paper_1908_11263_amd as qnn
    torch.cuda.set_device(0)
    qnn.device_check()
    graph = not args.no_graph

    if args.copy_bytes:
        a = torch.empty(args.copy_bytes, dtype=torch.uint8, device="cuda").fill_(1)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        log("copy calibration: %d bytes" % args.copy_bytes)

    if args.tile_sweep:
        tile_sweep(args)
        return

    workloads = {
        "int8": lambda: ConvStep(synth.int8_layer()),
        "int4": lambda: ConvStep(synth.int4_layer()),
        "int2": lambda: ConvStep(synth.int2_layer()),
        "int2_fp4": lambda: ConvStep(synth.int2_layer(), tile=(TILE_FP4, 0, 0, 0)),
        "int1": lambda: ConvStep(synth.int1_layer()),
        "int1_fp4": lambda: ConvStep(synth.int1_layer(), tile=(TILE_FP4, 0, 0, 0)),
        "int4_stair": lambda: ConvStep(synth.int4_stair_layer()),
        "cifar8": lambda: NetworkStep(synth.cifar_network(8, n=4096)),
        "cifar4": lambda: NetworkStep(synth.cifar_network(4, n=4096)),
    }
    head = "int4"
    names = [args.only] if args.only else [head] + [k for k in workloads if k != head]

    layers = {}
    for name in names:
        step = workloads[name]()
        steps = args.steps if name == head else max(20, min(args.steps, 200 if "cifar" in name else args.steps))
        warm = args.warmup if name == head else min(args.warmup, 10)
        log("workload %s: warmup %d, steps %d" % (name, warm, steps))
        sec, done = time_steps(step, steps, warm, graph=graph)
        gmacs = step.macs / sec / 1e9
        rec = {"macs_per_step": step.macs, "us_per_step": round(sec * 1e6, 3), "steps": done,
               "gmacs": round(gmacs, 2),
               "pct_int8_mfma_peak": round(100 * 2 * step.macs / sec / 1e12 / PEAK_INT8_TOPS, 3)}
        if name == "int2_fp4":
            rec["pct_fp4_mfma_peak"] = round(100 * 2 * step.macs / sec / 1e12 / PEAK_FP4_TFLOPS, 3)
        if name == "int1_fp4":
            rec["pct_fp4_mfma_peak"] = round(100 * 2 * step.macs / sec / 1e12 / PEAK_FP4_TFLOPS, 3)
        if name == "int1":
            rec["pct_xnor_valu_roofline"] = round(100 * step.macs / sec / XNOR_PEAK_BMACS, 3)
        if "cifar" in name:
            rec["images_per_s"] = round(step.net.n / sec, 1)
        if step.bytes:
            rec["algorithmic_gbs"] = round(step.bytes / sec / 1e9, 2)
        layers[name] = rec
        log("  %s: %.3f us/step, %.1f GMAC/s, %.2f%% of int8 MFMA peak"
            % (name, sec * 1e6, gmacs, rec["pct_int8_mfma_peak"]))
        if name == head:
            head_step, head_sec, head_done = step, sec, done
        else:
            del step
            torch.cuda.empty_cache()

    if head not in layers:
        return
    L = head_step.L
    achieved = 2 * head_step.macs / head_sec / 1e12
    traffic, kname = recorded_profile()
    roofline = {"bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_INT8_TOPS,
                "unit": "TOP/s", "frac": round(achieved / PEAK_INT8_TOPS, 5),
                "traffic": traffic, "kernel": kname or "conv_img_kernel<4, 32, 3, 3, 32, false, true> (row bands)",
                "ops_per_launch": 2 * head_step.macs}
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
                   "epilogue": "requant", "graph_replay": graph},
        "roofline": roofline,
        "layers": layers,
    }
    if not args.no_cpu and not args.only:
        log("cpu baseline (oracle) ...")
        out["cpu_baseline"] = cpu_baseline(L)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
