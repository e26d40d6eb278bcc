#!/usr/bin/env python3
"""Throughput of the parameterized fp32 GEMM / convolution path on one MI355X.

One step runs, once each and back to back on one stream:
  - the three 4096^3 GEMMs C = A op(B) + 0.5 C in the NN, TN and NT layouts;
  - the first conv layer of each VGG-16 block at batch 32 (3x3, stride 1,
    "same" padding): 224x224x3->64, 112x112x64->128, 56x56x128->256,
    28x28x256->512, 14x14x512->512;
  - five ResNet-50 bottleneck convolutions at batch 32: 56x56x64 1x1->64,
    3x3->64, 1x1->256; 56x56x256 1x1 stride 2->128; 7x7x2048 1x1->512.
All inputs are seeded synthetic fp32 values, uniform on [-1, 1), resident in
device memory before timing starts.  value = nominal flops of one step
(2*M*N*K per GEMM, 2*N*Ho*Wo*Cout*KH*KW*Cin per convolution) / time per step.

The timed region holds only its two end events.  Per-op durations come from
as many further steps with a fence-free HIP event before each launch, on the
launch stream (a default event between two kernels adds a system-scope cache
write-back to the span it closes).  The JSON line carries, for the kernel
launch with the largest share of the step, its fraction of the fp32 matrix
peak, the per-op figures, and the CPU oracle's rate on a bounded sample of the
same work.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "fp32 GFLOP/s & % of MI355X fp32 MFMA peak: GEMM 4096³, VGG/ResNet conv layers"
FP32_MFMA_PEAK_TFLOPS = 157.3   # 256 CUs x 256 flop/clk x 2.4 GHz
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target wall time of the CPU oracle sample (0 skips it)")
    ap.add_argument("--suite", default="step", choices=("step", "layers", "gemm-sweep", "winograd", "ablations",
                                                      "tune", "direct", "selector"),
                    help="step: the benchmark step (default); layers: every VGG-16 / ResNet-50 layer of the "
                         "paper at batch 1, 4 and 32; gemm-sweep: the paper's power-of-two GEMM sweep with "
                         "the vendor fp32 GEMM beside it; winograd: the 3x3 stride-1 layers through the "
                         "Winograd F(2x2, 3x3) and F(4x4, 3x3) paths beside the default path; ablations: double buffering, "
                         "vector width, wave-tile shape, tile size vs CU fill, operand loader, the convolution's "
                         "gather vs a dense operand, warm vs cold caches; tune: "
                         "the automated parameter search against the built-in choices; direct: every tiled "
                         "direct-convolution instance (tile x channel widths) on the small-channel layers; "
                         "selector: the rules' choice against the automated search on the paper's layers at "
                         "batch sizes the built-in table does not hold (2, 8, 12, 16)")
    ap.add_argument("--probes", action="store_true",
                    help="instead of the step: measure the fp32 MFMA rate (constant and random operands), "
                         "the HBM copy bandwidth and the vendor fp32 GEMM at 4096^3, print one JSON line")
    ap.add_argument("--text", action="store_true",
                    help="with --suite direct: print the tile x channel-width table instead of JSON")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="before timing, run one device-to-device copy of this many MiB (a kernel of "
                         "known traffic that scales the HBM byte counters)")
    return ap.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.txt")


def kernel_source_hash():
    """Hash of the HIP sources the benchmark step runs (the contraction and
    direct kernels, their instances and the selection that picks
    configuration and split): counters taken on other code no longer apply.
    The Winograd transforms and the probes are not part of the step."""
    import glob
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1904_05347_amd", "csrc")
    skip = {"pk_winograd.hip", "pk_probe.hip"}
    for path in sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.hpp"))):
        if os.path.basename(path) in skip:
            continue
        with open(path, "rb") as fh:
            h.update(os.path.basename(path).encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(op_name, config):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE
    summary, scaled by the copy-kernel calibration; None when that summary was
    taken on different kernel sources or lacks this launch."""
    try:
        with open(TRAFFIC_FILE) as fh:
            lines = fh.read().splitlines()
    except OSError:
        return None
    fields = dict(l.split(None, 1) for l in lines if l.startswith("source_hash "))
    if fields.get("source_hash", "").strip() != kernel_source_hash():
        return None
    for l in lines:
        if l.startswith("traffic |"):
            parts = [x.strip() for x in l.split("|")]
            if parts[1] == op_name and parts[2] == config:
                return int(parts[5])
    return None


class LightEvents:
    """HIP timing events created with hipEventDisableSystemFence, recorded on
    a given stream.  A default (torch) event between two kernels makes the
    next one wait for a system-scope cache write-back, about 6 us on MI355X,
    which is a large share of a 20-50 us layer; these events time the same
    stream-ordered span without it.  They use the HIP runtime already loaded
    in this process (the one torch and libpk.so share)."""

    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self):
        import ctypes
        path = None
        with open("/proc/self/maps") as fh:
            for line in fh:
                if "libamdhip64.so" in line:
                    path = line.split()[-1]
                    break
        if path is None:
            raise RuntimeError("no HIP runtime loaded in this process")
        self._ct = ctypes
        self._lib = ctypes.CDLL(path)
        self._lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        self._lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self._lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self._lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self._events = []

    def create(self):
        ev = self._ct.c_void_p()
        if self._lib.hipEventCreateWithFlags(self._ct.byref(ev), self.DISABLE_SYSTEM_FENCE) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")
        self._events.append(ev)
        return ev

    def record(self, ev, stream_handle):
        if self._lib.hipEventRecord(ev, self._ct.c_void_p(stream_handle)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_ms(self, e0, e1):
        ms = self._ct.c_float()
        if self._lib.hipEventElapsedTime(self._ct.byref(ms), e0, e1) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def close(self):
        for ev in self._events:
            self._lib.hipEventDestroy(ev)
        self._events = []


class Op:
    def __init__(self, name, flops, bytes_, run, kind):
        self.name = name
        self.flops = flops
        self.bytes = bytes_
        self.run = run
        self.kind = kind
        self.config = ""


def make_ops(torch, pk, wl):
    ops = []
    host = {}
    for case in wl.STEP_GEMMS:
        A, B, C = case.inputs()
        host[case.name] = ("gemm", case, (A, B, C))
        dA, dB, dC = (torch.from_numpy(v).cuda() for v in (A, B, C))
        ta, tb = case.trans_a == "T", case.trans_b == "T"

        def run(dA=dA, dB=dB, dC=dC, case=case, ta=ta, tb=tb):
            pk.gemm(dA, dB, dC, alpha=case.alpha, beta=case.beta, trans_a=ta, trans_b=tb)

        nbytes = 4 * (case.M * case.K + case.K * case.N + 2 * case.M * case.N)
        ops.append(Op(case.name, case.flops, nbytes, run, "gemm"))
    for case in wl.STEP_CONVS:
        x, f = case.inputs()
        host[case.name] = ("conv", case, (x, f))
        N, H, W, Cin = case.x_shape
        KH, KW, _, Cout = case.f_shape
        Ho, Wo = pk.conv2d_out_dims(H, W, KH, KW, *case.stride, *case.pads)
        dx, df = torch.from_numpy(x).cuda(), torch.from_numpy(f).cuda()
        dy = torch.empty((N, Ho, Wo, Cout), dtype=torch.float32, device="cuda")
        wsb = pk.conv2d_workspace_bytes(N, H, W, Cin, KH, KW, Cout, *case.stride, *case.pads)
        ws = torch.empty(wsb // 4, dtype=torch.float32, device="cuda") if wsb else None

        def run(dx=dx, df=df, dy=dy, ws=ws, case=case):
            pk.conv2d_fwd(dx, df, stride=case.stride, padding=case.pads, out=dy, workspace=ws)

        sh, sw = case.stride
        # input bytes the layer must read: every pixel for stride 1, the sampled ones otherwise
        in_px = N * (H if sh == 1 else Ho) * (W if sw == 1 else Wo) if KH == 1 and KW == 1 else N * H * W
        nbytes = 4 * (in_px * Cin + KH * KW * Cin * Cout + N * Ho * Wo * Cout)
        ops.append(Op(case.name, wl.conv_flops(case, Ho, Wo), nbytes, run, "conv"))
    return ops, host


def cpu_baseline(oracle, host, ops, seconds, np):
    """The oracle on the same fraction of every op's outputs, scaled to GFLOP/s."""
    rng = np.random.default_rng(2024)

    def run_fraction(frac):
        flops = 0
        n_out = 0
        t0 = time.perf_counter()
        for op in ops:
            kind, case, arrs = host[op.name]
            if kind == "gemm":
                A, B, C = arrs
                total = case.M * case.N
                n = max(1, int(round(total * frac)))
                flat = rng.integers(0, total, n)
                rows, cols = flat // case.N, flat % case.N
                oracle.sgemm_at(case.trans_a, case.trans_b, case.M, case.N, case.K, case.alpha,
                                A, case.lda, B, case.ldb, case.beta, C, case.ldc, rows, cols)
                flops += 2 * case.K * n
            else:
                x, f = arrs
                total = op.flops // (2 * case.KH * case.KW * case.Cin)
                n = max(1, int(round(total * frac)))
                flat = rng.integers(0, total, n)
                oracle.conv2d_at(x, f, case.stride, case.pads, flat)
                flops += 2 * case.KH * case.KW * case.Cin * n
            n_out += n
        return flops, n_out, time.perf_counter() - t0

    step_flops = sum(op.flops for op in ops)
    frac = 2e8 / step_flops  # calibration: about 0.2 GFLOP
    f0, _, t0 = run_fraction(frac)
    frac = min(frac * seconds / max(t0, 1e-3), 1.0)
    flops, n_out, t = run_fraction(frac)
    return {
        "value": round(flops / t / 1e9, 3),
        "unit": "GFLOP/s",
        "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": "%d outputs drawn uniformly from every op of one step (fraction %.3g of each op's "
                  "outputs, %.2f GFLOP nominal, fp64 accumulation), %.1f s" % (n_out, frac, flops / 1e9, t),
        "cpu_model": _cpu_model(),
        "per_core": per_core_baseline(oracle, np),
    }


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def per_core_baseline(oracle, np):
    """The oracle on one thread: the whole 512^3 GEMM and the whole batch-1
    56x56x64 -> 64 3x3 convolution (the two small parity workloads), GFLOP/s."""
    from paper_1904_05347_amd import workloads as wl
    threads = oracle.num_threads()
    oracle.set_threads(1)
    try:
        g = wl.GEMM_SMALL
        A, B, C = g.inputs()
        t0 = time.perf_counter()
        oracle.sgemm(g.trans_a, g.trans_b, g.M, g.N, g.K, g.alpha, A, g.lda, B, g.ldb, g.beta, C, g.ldc)
        tg = time.perf_counter() - t0
        c = wl.CONV_SMALL
        x, f = c.inputs()
        t0 = time.perf_counter()
        oracle.conv2d(x, f, c.stride, c.pads)
        tc = time.perf_counter() - t0
        Ho, Wo = c.out_hw
    finally:
        oracle.set_threads(threads)
    return {"threads": 1,
            "gemm_512_gflops": round(g.flops / tg / 1e9, 3),
            "conv_b1_56x56x64_gflops": round(wl.conv_flops(c, Ho, Wo) / tc / 1e9, 3)}


def _time_ms(torch, fn, min_ms=20.0):
    """Duration of fn on the current stream: after about 10 ms of untimed
    calls (so the clocks have left any idle state the host-side set-up let
    them fall into), three runs of back-to-back calls spanning about min_ms
    each; the median run's mean per call."""
    fn()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    fn()
    e1.record()
    torch.cuda.synchronize()
    one = max(e0.elapsed_time(e1), 1e-3)
    for _ in range(int(min(max(10.0 / one, 2), 400))):
        fn()
    iters = int(min(max(min_ms / one, 3), 200))
    runs = []
    for _ in range(3):
        e0.record()
        for _ in range(iters):
            fn()
        e1.record()
        torch.cuda.synchronize()
        runs.append(e0.elapsed_time(e1) / iters)
    return sorted(runs)[1]


def _time_ms_graph(torch, fn, calls=20, min_ms=20.0):
    """Device time of fn's kernels per call, without the host's per-call cost
    (a Python call through the binding takes about 10 us, longer than many
    small layers): `calls` calls captured into one HIP graph on a
    default-priority stream, the graph replayed for about 10 ms untimed, then
    three runs of replays spanning about min_ms each; the median run's mean
    per call."""
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(calls):
            fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    g.replay()
    e1.record()
    torch.cuda.synchronize()
    one = max(e0.elapsed_time(e1), 1e-3)
    for _ in range(int(min(max(10.0 / one, 2), 200))):
        g.replay()
    reps = int(min(max(min_ms / one, 3), 100))
    runs = []
    for _ in range(3):
        e0.record()
        for _ in range(reps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        runs.append(e0.elapsed_time(e1) / (reps * calls))
    del g
    return sorted(runs)[1]


def run_parity_configs(torch, pk, wl):
    """GEMM 512^3 (alpha 1, beta 0), the batch-1 56x56x64 3x3 convolution,
    and the 1024^3 and 2048^3 GEMMs (alpha 1, beta 0.5, C drawn after A and
    B): each with the default selection and the workspace the library asks
    for, device time per call from graph replay."""
    rows = []
    for case in (wl.GEMM_SMALL, wl.GEMM_SWEEP[0], wl.GEMM_SWEEP[1]):
        A, B, C = case.inputs()
        dA, dB, dC = (torch.from_numpy(v).cuda() for v in (A, B, C))
        ta, tb = case.trans_a == "T", case.trans_b == "T"
        need = pk.binding.sgemm_workspace_bytes(ta, tb, case.M, case.N, case.K)
        ws = torch.empty(max(need // 4, 1), dtype=torch.float32, device="cuda") if need else None

        def run(dA=dA, dB=dB, dC=dC, ws=ws, case=case, ta=ta, tb=tb):
            pk.gemm(dA, dB, dC, alpha=case.alpha, beta=case.beta, trans_a=ta, trans_b=tb, workspace=ws)

        ms = _time_ms_graph(torch, run)
        tf = case.flops / (ms * 1e-3) / 1e12
        rows.append({"op": case.name, "config": pk.last_config_name(), "alpha": case.alpha, "beta": case.beta,
                     "ms": round(ms, 5), "tflops": round(tf, 2),
                     "frac_mfma_peak": round(tf / FP32_MFMA_PEAK_TFLOPS, 4), "timing": "graph replay"})
        del dA, dB, dC, ws
    case = wl.CONV_SMALL
    x, f = case.inputs()
    N, H, W, Cin = case.x_shape
    KH, KW, _, Cout = case.f_shape
    Ho, Wo = pk.conv2d_out_dims(H, W, KH, KW, *case.stride, *case.pads)
    dx, df = torch.from_numpy(x).cuda(), torch.from_numpy(f).cuda()
    dy = torch.empty((N, Ho, Wo, Cout), dtype=torch.float32, device="cuda")
    wsb = pk.conv2d_workspace_bytes(N, H, W, Cin, KH, KW, Cout, *case.stride, *case.pads)
    ws = torch.empty(wsb // 4, dtype=torch.float32, device="cuda") if wsb else None

    def run():
        pk.conv2d_fwd(dx, df, stride=case.stride, padding=case.pads, out=dy, workspace=ws)

    ms = _time_ms_graph(torch, run)
    tf = wl.conv_flops(case, Ho, Wo) / (ms * 1e-3) / 1e12
    rows.append({"op": case.name, "config": pk.last_config_name(), "ms": round(ms, 5), "tflops": round(tf, 2),
                 "frac_mfma_peak": round(tf / FP32_MFMA_PEAK_TFLOPS, 4), "timing": "graph replay"})
    return rows


def run_layer_suite(torch, pk, wl):
    """Every distinct layer of the paper's VGG-16 / ResNet-50 tables at batch 1, 4, 32."""
    rows = []
    for batch in (1, 4, 32):
        for case in wl.layer_suite(batch):
            x, f = case.inputs()
            N, H, W, Cin = case.x_shape
            KH, KW, _, Cout = case.f_shape
            Ho, Wo = pk.conv2d_out_dims(H, W, KH, KW, *case.stride, *case.pads)
            dx, df = torch.from_numpy(x).cuda(), torch.from_numpy(f).cuda()
            dy = torch.empty((N, Ho, Wo, Cout), dtype=torch.float32, device="cuda")
            wsb = pk.conv2d_workspace_bytes(N, H, W, Cin, KH, KW, Cout, *case.stride, *case.pads)
            ws = torch.empty(wsb // 4, dtype=torch.float32, device="cuda") if wsb else None

            def run():
                pk.conv2d_fwd(dx, df, stride=case.stride, padding=case.pads, out=dy, workspace=ws)

            ms = _time_ms_graph(torch, run)
            flops = wl.conv_flops(case, Ho, Wo)
            nbytes = 4 * (x.size + f.size + N * Ho * Wo * Cout)
            rows.append({"layer": case.name, "config": pk.last_config_name(), "ms": round(ms, 4),
                         "tflops": round(flops / (ms * 1e-3) / 1e12, 2),
                         "frac_mfma_peak": round(flops / (ms * 1e-3) / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4),
                         "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
                         "flop_per_byte": round(flops / nbytes, 1)})
            del dx, df, dy, ws
            print("bench: %s %.4f ms" % (case.name, ms), file=sys.stderr, flush=True)
    return {"suite": "layers", "dtype": "f32", "data": "synthetic", "rows": rows}


def run_direct_suite(torch, pk, wl):
    """The tiled direct convolution's parameter space (Section 4.1.1: output
    tile x output- and input-channel widths) on the paper's small-channel
    first layers and a 3x3 layer with 16 input channels, at batch 32 (and the
    first layers at 1 and 4): every instance that takes the layer, forced,
    graph-timed, beside the default selection.  Rows carry the tile (rows x
    columns), the channel widths and TFLOP/s, the data of the heatmap."""
    layers = [c for c in wl.layer_suite(32) if c.x_shape[3] == 3]
    layers += [c for b in (1, 4) for c in wl.layer_suite(b) if c.x_shape[3] == 3]
    layers.append(wl.ConvCase("synthetic b32 56x56x16->64 3x3 s1", 32, 56, 56, 16, 3, 3, 64, (1, 1),
                              (1, 1, 1, 1), 77, (56, 56)))
    tiled = [c for c in pk.configs() if c["kind"] == 2]
    rows = []
    for case in layers:
        x, f = case.inputs()
        N, H, W, Cin = case.x_shape
        KH, KW, _, Cout = case.f_shape
        Ho, Wo = pk.conv2d_out_dims(H, W, KH, KW, *case.stride, *case.pads)
        dx, df = torch.from_numpy(x).cuda(), torch.from_numpy(f).cuda()
        dy = torch.empty((N, Ho, Wo, Cout), dtype=torch.float32, device="cuda")
        flops = wl.conv_flops(case, Ho, Wo)
        wsb = pk.conv2d_workspace_bytes(N, H, W, Cin, KH, KW, Cout, *case.stride, *case.pads)
        ws = torch.empty(wsb // 4, dtype=torch.float32, device="cuda") if wsb else None
        ms = _time_ms_graph(torch, lambda: pk.conv2d_fwd(dx, df, stride=case.stride, padding=case.pads, out=dy,
                                                         workspace=ws))
        rows.append({"layer": case.name, "config": pk.last_config_name(), "variant": "default", "ms": round(ms, 4),
                     "tflops": round(flops / (ms * 1e-3) / 1e12, 2)})
        for cfg in tiled:
            pk.force_config(cfg["name"])
            try:
                pk.conv2d_fwd(dx, df, stride=case.stride, padding=case.pads, out=dy)
            except pk.PkError:
                pk.force_config(None)
                continue
            try:
                ms = _time_ms_graph(torch, lambda: pk.conv2d_fwd(dx, df, stride=case.stride, padding=case.pads,
                                                                 out=dy))
            finally:
                pk.force_config(None)
            rows.append({"layer": case.name, "config": cfg["name"], "variant": "forced", "ms": round(ms, 4), "tflops": round(flops / (ms * 1e-3) / 1e12, 2),
                         "frac_mfma_peak": round(flops / (ms * 1e-3) / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4)})
            print("bench: %s %s %.4f ms" % (case.name, cfg["name"], ms), file=sys.stderr, flush=True)
        del dx, df, dy, ws
    return {"suite": "direct", "dtype": "f32", "data": "synthetic", "rows": rows}


def direct_heatmap(result):
    """The direct suite as text: per layer, one row per output tile
    (rows x columns of a work-group) and one column per (output channels,
    input-channel load width v1 / v4, or tp: the persistent form with
    double-buffered patches), TFLOP/s in the cells; the default selection
    and the fixed-tile kernels below."""
    import re
    out = []
    layers = []
    for r in result["rows"]:
        if r["layer"] not in layers:
            layers.append(r["layer"])
    for layer in layers:
        rows = [r for r in result["rows"] if r["layer"] == layer]
        cells, other = {}, []
        for r in rows:
            m = re.match(r"direct_(\d+)x(\d+)x(\d+)_(v\d+|tp)$", r["config"])
            if r["variant"] == "forced" and m:
                tr, tc, ch = (int(v) for v in m.groups()[:3])
                cells[(tr, tc), (ch, m.group(4))] = r["tflops"]
            else:
                other.append("  %s %s: %.4f ms, %.2f TFLOP/s" % (r["variant"], r["config"], r["ms"], r["tflops"]))
        cols = sorted({c for _, c in cells})
        tiles = sorted({t for t, _ in cells})
        out.append(layer)
        out.append("  %-10s" % "tile" + "".join("  ch%-3d %-2s" % c for c in cols))
        for t in tiles:
            out.append("  %-10s" % ("%dx%d" % t) +
                       "".join(("%9.1f" % cells[t, c]) if (t, c) in cells else "%9s" % "-" for c in cols))
        out.extend(other)
        out.append("")
    return "\n".join(out)


def run_winograd_suite(torch, pk, wl):
    """Every 3x3 stride-1 layer of the paper's tables at batch 1, 4, 32: the
    Winograd path with output tiles of 2 x 2 (F(2x2, 3x3)) and of 4 x 4
    (F(4x4, 3x3)) beside the default (implicit-GEMM) path.  TFLOP/s are
    nominal (the direct sum's 2*N*Ho*Wo*Cout*9*Cin over the time);
    product_tflops counts the (m+2)^2 batched products each Winograd form
    runs."""
    rows = []
    for batch in (1, 4, 32):
        for case in wl.layer_suite(batch):
            KH, KW, Cin, Cout = case.f_shape
            if (KH, KW) != (3, 3) or case.stride != (1, 1):
                continue
            x, f = case.inputs()
            N, H, W, _ = case.x_shape
            Ho, Wo = pk.conv2d_out_dims(H, W, 3, 3, 1, 1, *case.pads)
            dx, df = torch.from_numpy(x).cuda(), torch.from_numpy(f).cuda()
            dy = torch.empty((N, Ho, Wo, Cout), dtype=torch.float32, device="cuda")
            wsb = pk.conv2d_workspace_bytes(N, H, W, Cin, 3, 3, Cout, 1, 1, *case.pads)
            ws = torch.empty(wsb // 4, dtype=torch.float32, device="cuda") if wsb else None
            ms_d = _time_ms_graph(torch, lambda: pk.conv2d_fwd(dx, df, padding=case.pads, out=dy, workspace=ws))
            cfg_d = pk.last_config_name()
            flops = wl.conv_flops(case, Ho, Wo)
            row = {"layer": case.name, "config_direct": cfg_d, "ms_direct": round(ms_d, 4),
                   "tflops_direct": round(flops / (ms_d * 1e-3) / 1e12, 2)}
            for m in (2, 4):
                wwb = pk.conv2d_winograd_workspace_bytes(N, H, W, Cin, Cout, *case.pads, m)
                wws = torch.empty(wwb // 4, dtype=torch.float32, device="cuda")
                ms_w = _time_ms_graph(torch, lambda: pk.conv2d_winograd(dx, df, padding=case.pads, out=dy,
                                                                        workspace=wws, tile=m))
                tiles = N * ((Ho + m - 1) // m) * ((Wo + m - 1) // m)
                prod_flops = (m + 2) ** 2 * 2 * tiles * Cin * Cout
                row.update({"config_f%d" % m: pk.last_config_name(), "ms_f%d" % m: round(ms_w, 4),
                            "speedup_f%d" % m: round(ms_d / ms_w, 3),
                            "tflops_nominal_f%d" % m: round(flops / (ms_w * 1e-3) / 1e12, 2),
                            "product_tflops_f%d" % m: round(prod_flops / (ms_w * 1e-3) / 1e12, 2),
                            "workspace_mib_f%d" % m: round(wwb / 2 ** 20, 1)})
                del wws
            rows.append(row)
            del dx, df, dy, ws
            print("bench: %s direct %.4f ms F2 %.4f ms F4 %.4f ms" % (case.name, ms_d, row["ms_f2"], row["ms_f4"]),
                  file=sys.stderr, flush=True)
    return {"suite": "winograd", "dtype": "f32", "data": "synthetic", "rows": rows}


def _time_each(torch, fn, iters=50, between=None):
    """Median and minimum (ms) of `iters` individually timed calls, each
    bracketed by HIP events on the current stream; `between` runs untimed
    before each call (e.g. a scratch write that evicts the caches)."""
    fn()
    fn()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    times = []
    for _ in range(iters):
        if between is not None:
            between()
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    times.sort()
    return times[len(times) // 2], times[0]


def run_ablations(torch, pk, wl):
    """The design choices the paper varies, measured on MI355X: double
    buffering (two LDS stages vs one), load vector width (16/8/4 bytes),
    square vs elongated wave tiles at equal accumulator count, tile size
    against CU fill, the operand loader (register-staged vs copied straight
    into LDS, and the direct copies' stage count), the convolution's gather
    against a dense operand of the same shape, and warm vs cold caches for
    the layers whose working set fits the 256 MB last-level cache.  Median
    and min of 50 individually timed calls each."""
    import numpy as np

    rows = []

    def gemm_rows(ablation, case, variants):
        A, B, C = case.inputs()
        dA, dB, dC = (torch.from_numpy(v).cuda() for v in (A, B, C))
        for label, cfg in variants:
            pk.force_config(cfg)
            try:
                med, mn = _time_each(torch, lambda: pk.gemm(dA, dB, dC, alpha=case.alpha, beta=case.beta))
                used = pk.last_config_name()
            finally:
                pk.force_config(None)
            c = next(x for x in pk.configs() if x["name"] == cfg)
            tiles = -(-case.M // c["bm"]) * -(-case.N // c["bn"])
            rows.append({"ablation": ablation, "shape": case.name, "variant": label, "config": used,
                         "ms_median": round(med, 4), "ms_min": round(mn, 4),
                         "tflops": round(case.flops / (med * 1e-3) / 1e12, 2), "tiles": tiles,
                         "tiles_per_cu": round(tiles / 256, 2)})
            print("bench: %s %s %s %.4f ms" % (ablation, case.name, label, med), file=sys.stderr, flush=True)
        del dA, dB, dC

    g1024, g2048, g4096 = wl.GEMM_SWEEP[0], wl.GEMM_SWEEP[1], wl.GEMM_SWEEP[2]
    for case in (g4096, g1024):
        gemm_rows("double buffering", case, [
            ("two LDS stages 128x128x16", "gemm_128x128x16_w2x2_nn_v44"),
            ("one LDS stage 128x128x16", "gemm_128x128x16_w2x2_nn_v44_s1"),
            ("two LDS stages 64x64x32", "gemm_64x64x32_w2x2_nn_v44"),
            ("one LDS stage 64x64x32", "gemm_64x64x32_w2x2_nn_v44_s1"),
            ("two LDS stages 256x256x32", "gemm_256x256x32_w2x4_nn_v44_o2"),
            ("one LDS stage 256x256x32", "gemm_256x256x32_w2x4_nn_v44_o2_s1")])
        gemm_rows("vector width", case, [
            ("16-byte loads", "gemm_128x128x16_w2x2_nn_v44"),
            ("8-byte loads", "gemm_128x128x16_w2x2_nn_v22"),
            ("4-byte loads", "gemm_128x128x16_w2x2_nn_v11")])
        gemm_rows("wave tile shape", case, [
            ("64x64 per wave (square)", "gemm_128x128x16_w2x2_nn_v44"),
            ("32x128 per wave", "gemm_128x128x16_w4x1_nn_v44"),
            ("128x32 per wave", "gemm_128x128x16_w1x4_nn_v44")])
    for case in (g1024, g2048, g4096):
        gemm_rows("tile size vs CU fill", case, [
            ("64x64 tiles", "gemm_64x64x32_w2x2_nn_v44"),
            ("128x128 tiles", "gemm_128x128x32_w2x2_nn_v44"),
            ("256x256 tiles", "gemm_256x256x32_w2x4_nn_v44_o2"),
            ("128x128 tiles, persistent", "gemm_128x128x32_w2x4_nn_v44_o2_p")])

    # operand staging: global -> registers -> LDS (ds_write) against global ->
    # LDS directly (buffer_load ... lds), same tile and MFMA pipeline
    gemm_rows("operand loader", g4096, [
        ("register-staged 256x256x32", "gemm_256x256x32_w2x4_nn_v44_o2"),
        ("direct-to-LDS 256x256x32, 2 stages", "gemm_256x256x32_w2x4_nn_v44_o2_dma2"),
        ("register-staged 128x128x16", "gemm_128x128x16_w2x2_nn_v44"),
        ("direct-to-LDS 128x128x16, 3 stages", "gemm_128x128x16_w2x2_nn_v44_dma3"),
        ("register-staged 64x64x32", "gemm_64x64x32_w2x2_nn_v44"),
        ("direct-to-LDS 64x64x32, 3 stages", "gemm_64x64x32_w2x2_nn_v44_dma3")])
    gemm_rows("direct-to-LDS stages", g4096, [
        ("2 stages 256x256x16", "gemm_256x256x16_w2x4_nn_v44_o2_dma2"),
        ("3 stages 256x256x16", "gemm_256x256x16_w2x4_nn_v44_o2_dma3"),
        ("4 stages 256x256x16", "gemm_256x256x16_w2x4_nn_v44_o2_dma4")])
    by_name = {c.name: c for c in wl.STEP_CONVS}
    for name, variants in (
            ("vgg16 conv2_1 b32 112x112x64->128 3x3", [
                ("register-staged 128x128x32", "conv_128x128x32_w2x4_v44_o2"),
                ("direct-to-LDS 128x128x32, 2 stages", "conv_128x128x32_w2x4_v44_o2_dma2")]),
            ("vgg16 conv3_1 b32 56x56x128->256 3x3", [
                ("register-staged 128x128x32, stream-K", "conv_128x128x32_w2x4_v44_o2_sk"),
                ("direct-to-LDS 128x128x32, stream-K", "conv_128x128x32_w2x4_v44_o2_dma2_sk")])):
        case = by_name[name]
        x, f = case.inputs()
        N, H, W, Cin = case.x_shape
        KH, KW, _, Cout = case.f_shape
        Ho, Wo = case.out_hw
        dx, df = torch.from_numpy(x).cuda(), torch.from_numpy(f).cuda()
        dy = torch.empty((N, Ho, Wo, Cout), dtype=torch.float32, device="cuda")
        ws = torch.empty(64 << 20, dtype=torch.float32, device="cuda")
        for label, cfg in variants:
            pk.force_config(cfg)
            try:
                med, mn = _time_each(torch, lambda: pk.conv2d_fwd(dx, df, stride=case.stride, padding=case.pads,
                                                                  out=dy, workspace=ws))
                used = pk.last_config_name()
            finally:
                pk.force_config(None)
            rows.append({"ablation": "operand loader", "shape": name, "variant": label, "config": used,
                         "ms_median": round(med, 4), "ms_min": round(mn, 4),
                         "tflops": round(wl.conv_flops(case, Ho, Wo) / (med * 1e-3) / 1e12, 2)})
            print("bench: operand loader %s %s %.4f ms" % (name, label, med), file=sys.stderr, flush=True)
        del dx, df, dy, ws

    # what the convolution's gather costs: each VGG layer against a dense NN
    # GEMM of its implicit-GEMM shape (M = N*Ho*Wo, N = Cout, K = KH*KW*Cin)
    # on the same tile and pipeline, and the same layer on 256x256 tiles
    for name, forms in (
            ("vgg16 conv2_1 b32 112x112x64->128 3x3", [
                ("128x128x32, 2 stages", "conv_128x128x32_w2x4_v44_o2_dma2", "gemm_128x128x32_w2x4_nn_v44_o2_dma2"),
                ("256x256x32, 2 stages", "conv_256x256x32_w2x4_v44_o2_dma2", "gemm_256x256x32_w2x4_nn_v44_o2_dma2")]),
            ("vgg16 conv4_1 b32 28x28x256->512 3x3", [
                ("128x128x32, stream-K", "conv_128x128x32_w2x4_v44_o2_dma2_sk",
                 "gemm_128x128x32_w2x4_nn_v44_o2_dma2_sk"),
                ("256x256x32, 2 stages", "conv_256x256x32_w2x4_v44_o2_dma2", "gemm_256x256x32_w2x4_nn_v44_o2_dma2")])):
        case = by_name[name]
        x, f = case.inputs()
        N, H, W, Cin = case.x_shape
        KH, KW, _, Cout = case.f_shape
        Ho, Wo = case.out_hw
        M, K = N * Ho * Wo, KH * KW * Cin
        rng = np.random.default_rng(M + K)
        dx, df = torch.from_numpy(x).cuda(), torch.from_numpy(f).cuda()
        dy = torch.empty((N, Ho, Wo, Cout), dtype=torch.float32, device="cuda")
        dA = torch.from_numpy(wl.uniform(rng, M * K).reshape(M, K)).cuda()
        dB = torch.from_numpy(wl.uniform(rng, K * Cout).reshape(K, Cout)).cuda()
        dC = torch.empty((M, Cout), dtype=torch.float32, device="cuda")
        ws = torch.empty(64 << 20, dtype=torch.float32, device="cuda")
        fl = wl.conv_flops(case, Ho, Wo)
        for label, conv_cfg, gemm_cfg in forms:
            for what, cfg, fn in (
                    ("convolution (gathered A)", conv_cfg,
                     lambda: pk.conv2d_fwd(dx, df, stride=case.stride, padding=case.pads, out=dy, workspace=ws)),
                    ("dense GEMM %dx%dx%d" % (M, Cout, K), gemm_cfg, lambda: pk.gemm(dA, dB, dC, workspace=ws))):
                pk.force_config(cfg)
                try:
                    med, mn = _time_each(torch, fn)
                    used = pk.last_config_name()
                finally:
                    pk.force_config(None)
                rows.append({"ablation": "gather vs dense A", "shape": name, "variant": "%s, %s" % (what, label),
                             "config": used, "ms_median": round(med, 4), "ms_min": round(mn, 4),
                             "tflops": round(fl / (med * 1e-3) / 1e12, 2)})
                print("bench: gather vs dense %s %s %s %.4f ms" % (name, what, label, med), file=sys.stderr,
                      flush=True)
        del dx, df, dy, dA, dB, dC, ws

    # the 4096^2-output GEMM's K loop against its fixed per-call part: the
    # same configuration at three depths, with and without the read of C
    rng = np.random.default_rng(4096)
    dA = torch.from_numpy(wl.uniform(rng, 4096 * 4096).reshape(4096, 4096)).cuda()
    dB = torch.from_numpy(wl.uniform(rng, 4096 * 4096).reshape(4096, 4096)).cuda()
    dC = torch.from_numpy(wl.uniform(rng, 4096 * 4096).reshape(4096, 4096)).cuda()
    cfg = "gemm_256x256x32_w2x4_nn_v44_o2_dma2"
    for k in (1024, 2048, 4096):
        Ak, Bk = dA[:, :k].contiguous(), dB[:k].contiguous()
        for beta in (0.0, 0.5):
            pk.force_config(cfg)
            try:
                med, mn = _time_each(torch, lambda: pk.gemm(Ak, Bk, dC, beta=beta))
                used = pk.last_config_name()
            finally:
                pk.force_config(None)
            rows.append({"ablation": "K loop vs fixed part", "shape": "gemm NN 4096x4096x%d" % k,
                         "variant": "beta = %g" % beta, "config": used, "ms_median": round(med, 4),
                         "ms_min": round(mn, 4), "tflops": round(2.0 * 4096 * 4096 * k / (med * 1e-3) / 1e12, 2)})
            print("bench: K loop %d beta %g %.4f ms" % (k, beta, med), file=sys.stderr, flush=True)
        del Ak, Bk
    del dA, dB, dC

    # warm vs cold: a 512 MiB scratch write between calls evicts L2 and MALL
    scratch = torch.empty(128 << 20, dtype=torch.float32, device="cuda")
    for name in ("vgg16 conv1_1 b32 224x224x3->64 3x3", "resnet50 b32 56x56x64->64 1x1",
                 "resnet50 b32 56x56x64->256 1x1"):
        case = by_name[name]
        x, f = case.inputs()
        N, H, W, Cin = case.x_shape
        KH, KW, _, Cout = case.f_shape
        Ho, Wo = case.out_hw
        dx, df = torch.from_numpy(x).cuda(), torch.from_numpy(f).cuda()
        dy = torch.empty((N, Ho, Wo, Cout), dtype=torch.float32, device="cuda")
        nbytes = 4 * (x.size + f.size + dy.numel())

        def run():
            pk.conv2d_fwd(dx, df, stride=case.stride, padding=case.pads, out=dy)

        # device time from graph replay: warm = 20 calls back to back; cold =
        # 20 x (512 MiB write, call) minus 20 x (512 MiB write) alone
        def evict():
            scratch.fill_(1.0)

        def evict_and_run():
            scratch.fill_(1.0)
            run()

        warm = _time_ms_graph(torch, run)
        cold = _time_ms_graph(torch, evict_and_run) - _time_ms_graph(torch, evict)
        for label, ms in (("warm", warm), ("cold (512 MiB write before each call)", cold)):
            rows.append({"ablation": "cache state", "shape": name, "variant": label, "config": pk.last_config_name(),
                         "ms_median": round(ms, 4), "timing": "graph replay",
                         "tflops": round(wl.conv_flops(case, Ho, Wo) / (ms * 1e-3) / 1e12, 2),
                         "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1)})
            print("bench: cache %s %s %.4f ms" % (name, label, ms), file=sys.stderr, flush=True)
        del dx, df, dy
    return {"suite": "ablations", "dtype": "f32", "data": "synthetic", "rows": rows}


def run_tune_suite(torch, pk, wl):
    """The automated parameter search against the built-in choices: for the
    benchmark step's ops and every layer of the paper's tables at batch 4,
    the default configuration's time, then pk_tune_* on the same operands,
    then the recorded choice's time (back-to-back timing as in the layer
    suite)."""
    rows = []
    pk.tune_reset()
    for case in wl.STEP_GEMMS:
        A, B, C = case.inputs()
        dA, dB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
        dC = torch.from_numpy(C).cuda()
        ta, tb = case.trans_a == "T", case.trans_b == "T"

        def run():
            pk.gemm(dA, dB, dC, alpha=case.alpha, beta=case.beta, trans_a=ta, trans_b=tb)

        ms0 = _time_ms(torch, run)
        cfg0 = pk.last_config_name()
        scratch = torch.empty_like(dC)
        r = pk.tune_gemm(dA, dB, scratch, alpha=case.alpha, beta=case.beta, trans_a=ta, trans_b=tb, iters=5)
        ms1 = _time_ms(torch, run)
        rows.append({"op": case.name, "default": cfg0, "default_ms": round(ms0, 4), "tuned": r["config"],
                     "tuned_splits": r["splits"], "tuned_ms": round(ms1, 4), "candidates": r["candidates"],
                     "speedup": round(ms0 / ms1, 3)})
        print("bench: tune %s %s -> %s %.3fx" % (case.name, cfg0, r["config"], ms0 / ms1), file=sys.stderr, flush=True)
        del dA, dB, dC, scratch
    for case in list(wl.STEP_CONVS) + list(wl.layer_suite(4)):
        x, f = case.inputs()
        N, H, W, Cin = case.x_shape
        KH, KW, _, Cout = case.f_shape
        if KH != KW or case.stride[0] != case.stride[1]:
            continue
        Ho, Wo = pk.conv2d_out_dims(H, W, KH, KW, *case.stride, *case.pads)
        dx, df = torch.from_numpy(x).cuda(), torch.from_numpy(f).cuda()
        dy = torch.empty((N, Ho, Wo, Cout), dtype=torch.float32, device="cuda")
        # room for the default rule's split and for every split the tuner tries
        wsb = pk.conv2d_workspace_bytes(N, H, W, Cin, KH, KW, Cout, *case.stride, *case.pads)
        ws = torch.empty(max(8 * N * Ho * Wo * Cout, wsb // 4), dtype=torch.float32, device="cuda")

        def run():
            pk.conv2d_fwd(dx, df, stride=case.stride, padding=case.pads, out=dy, workspace=ws)

        ms0 = _time_ms(torch, run)
        cfg0 = pk.last_config_name()
        r = pk.tune_conv2d(dx, df, stride=case.stride, padding=case.pads, out=dy, workspace=ws, iters=3)
        ms1 = _time_ms(torch, run)
        rows.append({"op": case.name, "default": cfg0, "default_ms": round(ms0, 4), "tuned": r["config"],
                     "tuned_splits": r["splits"], "tuned_ms": round(ms1, 4), "candidates": r["candidates"],
                     "speedup": round(ms0 / ms1, 3)})
        print("bench: tune %s %s -> %s/%d %.3fx" % (case.name, cfg0, r["config"], r["splits"], ms0 / ms1),
              file=sys.stderr, flush=True)
        del dx, df, dy, ws
    pk.tune_reset()
    return {"suite": "tune", "dtype": "f32", "data": "synthetic", "rows": rows}


def run_selector_suite(torch, pk, wl, batches=(2, 8, 12, 16)):
    """How the selection rules generalise: every layer of the paper's tables
    (square windows and strides) at batch sizes the built-in table does not
    hold, timed with the rules' choice, then with the automated search's
    choice (pk_tune_conv2d_fwd on the same operands, splits up to 16), both
    by graph replay; the ratio of the two times is what the rules leave on
    the table for shapes nobody measured."""
    rows = []
    for batch in batches:
        for case in wl.layer_suite(batch):
            N, H, W, Cin = case.x_shape
            KH, KW, _, Cout = case.f_shape
            if KH != KW or case.stride[0] != case.stride[1]:
                continue
            x, f = case.inputs()
            Ho, Wo = pk.conv2d_out_dims(H, W, KH, KW, *case.stride, *case.pads)
            dx, df = torch.from_numpy(x).cuda(), torch.from_numpy(f).cuda()
            dy = torch.empty((N, Ho, Wo, Cout), dtype=torch.float32, device="cuda")
            wsb = pk.conv2d_workspace_bytes(N, H, W, Cin, KH, KW, Cout, *case.stride, *case.pads)
            ws = torch.empty(max(wsb // 4, 1), dtype=torch.float32, device="cuda")
            pk.tune_reset()
            ms_r = _time_ms_graph(torch, lambda: pk.conv2d_fwd(dx, df, stride=case.stride, padding=case.pads,
                                                              out=dy, workspace=ws))
            cfg_r = pk.last_config_name()
            wst = torch.empty(min(16 * N * Ho * Wo * Cout, 1 << 29), dtype=torch.float32, device="cuda")
            r = pk.tune_conv2d(dx, df, stride=case.stride, padding=case.pads, out=dy, workspace=wst, iters=3)
            ms_s = _time_ms_graph(torch, lambda: pk.conv2d_fwd(dx, df, stride=case.stride, padding=case.pads,
                                                              out=dy, workspace=wst))
            pk.tune_reset()
            rows.append({"layer": case.name, "rules": cfg_r, "ms_rules": round(ms_r, 4), "search": r["config"],
                         "search_splits": r["splits"], "ms_search": round(ms_s, 4),
                         "rules_over_search": round(ms_r / ms_s, 3)})
            print("bench: %s rules %s %.4f ms, search %s/%d %.4f ms" % (case.name, cfg_r, ms_r, r["config"],
                  r["splits"], ms_s), file=sys.stderr, flush=True)
            del dx, df, dy, ws, wst
    return {"suite": "selector", "dtype": "f32", "data": "synthetic", "rows": rows}


def run_gemm_sweep(torch, pk, wl):
    """The paper's GEMM sweep (M, N, K powers of two in [64, 1024]), with the
    vendor fp32 GEMM (torch.matmul, tf32 off) timed beside it as context."""
    torch.backends.cuda.matmul.allow_tf32 = False
    rows = []
    for case in wl.gemm_sweep():
        A, B, C = case.inputs()
        dA, dB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
        dC = torch.empty((case.M, case.N), dtype=torch.float32, device="cuda")
        ms = _time_ms_graph(torch, lambda: pk.gemm(dA, dB, dC))
        cfg = pk.last_config_name()
        ms_v = _time_ms_graph(torch, lambda: torch.matmul(dA, dB, out=dC))
        nbytes = 4 * (case.M * case.K + case.K * case.N + case.M * case.N)
        rows.append({"M": case.M, "N": case.N, "K": case.K, "config": cfg,
                     "flop_per_byte": round(case.flops / nbytes, 2),
                     "gflops": round(case.flops / (ms * 1e-3) / 1e9, 1),
                     "vendor_gflops": round(case.flops / (ms_v * 1e-3) / 1e9, 1)})
    return {"suite": "gemm-sweep", "dtype": "f32", "data": "synthetic", "rows": rows}


def run_probes(torch, pk):
    """Denominators measured on this GPU, and the vendor fp32 GEMM as context."""
    from paper_1904_05347_amd import binding
    warm = torch.rand(4096, 4096, device="cuda")
    for _ in range(40):
        pk.gemm(warm, warm)
    torch.cuda.synchronize()
    out = {"mfma_const_operands_tflops": {}, "mfma_random_operands_tflops": {}}
    for blocks in (768, 2048):  # 768 = one round of 3 work-groups per CU
        out["mfma_const_operands_tflops"][blocks] = round(binding.probe_mfma_peak_tflops(blocks, 8000), 2)
        out["mfma_random_operands_tflops"][blocks] = round(binding.probe_mfma_data_tflops(blocks, 2000), 2)
    out["copy_gbs_2GiB"] = round(binding.probe_copy_gbs(2048), 1)
    torch.backends.cuda.matmul.allow_tf32 = False
    a = torch.rand(4096, 4096, device="cuda") * 2 - 1
    b = torch.rand(4096, 4096, device="cuda") * 2 - 1
    for _ in range(3):
        a @ b
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(10):
        a @ b
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 10
    out["vendor_fp32_gemm_4096_tflops"] = round(2 * 4096 ** 3 / (ms * 1e-3) / 1e12, 2)
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (requested --gpus %d)" % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_1904_05347_amd as pk
    from paper_1904_05347_amd import workloads as wl

    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    pk.load()
    if args.probes:
        print(json.dumps(run_probes(torch, pk)))
        return
    if args.suite == "layers":
        print(json.dumps(run_layer_suite(torch, pk, wl)))
        return
    if args.suite == "gemm-sweep":
        print(json.dumps(run_gemm_sweep(torch, pk, wl)))
        return
    if args.suite == "winograd":
        print(json.dumps(run_winograd_suite(torch, pk, wl)))
        return
    if args.suite == "ablations":
        print(json.dumps(run_ablations(torch, pk, wl)))
        return
    if args.suite == "direct":
        res = run_direct_suite(torch, pk, wl)
        print(direct_heatmap(res) if args.text else json.dumps(res))
        return
    if args.suite == "selector":
        print(json.dumps(run_selector_suite(torch, pk, wl)))
        return
    if args.suite == "tune":
        print(json.dumps(run_tune_suite(torch, pk, wl)))
        return
    print("bench: generating inputs", file=sys.stderr, flush=True)
    ops, host = make_ops(torch, pk, wl)
    stream = torch.cuda.current_stream()
    if args.copy_probe_mib > 0:
        n = args.copy_probe_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # one untimed pass records which configuration each op runs
    for op in ops:
        op.run()
        op.config = pk.last_config_name()
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        for op in ops:
            op.run()
    torch.cuda.synchronize()
    print("bench: warmed up, timing %d steps" % args.steps, file=sys.stderr, flush=True)

    # the timed region: K steps back to back, events only at its two ends
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for s in range(args.steps):
        for op in ops:
            op.run()
    end.record(stream)
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(end) / args.steps
    step_flops = sum(op.flops for op in ops)
    value = step_flops / (ms_per_step * 1e-3) / 1e9

    # per-op durations: K more steps with a fence-free HIP event before each
    # op, on the stream the kernels are launched on
    print("bench: timing each op inside %d more steps" % args.steps, file=sys.stderr, flush=True)
    light = LightEvents()
    handle = stream.cuda_stream
    ev = [[light.create() for _ in range(len(ops) + 1)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    for s in range(args.steps):
        for i, op in enumerate(ops):
            light.record(ev[s][i], handle)
            op.run()
        light.record(ev[s][len(ops)], handle)
    torch.cuda.synchronize()
    ms_per_step_with_op_events = light.elapsed_ms(ev[0][0], ev[-1][len(ops)]) / args.steps

    # context figures of this GPU, measured after the timed region: an MFMA
    # issue probe (random operands, not a ceiling: the 4096^3 GEMMs exceed
    # it) and a 16-byte streaming copy
    from paper_1904_05347_amd import binding
    measured = {"mfma_random_operands_probe_tflops": round(binding.probe_mfma_data_tflops(768, 2000), 2),
                "copy_gbs": round(binding.probe_copy_gbs(1024), 1)}

    # the parity configurations at their stated alpha / beta, with the default
    # selection and the workspace the library asks for (outside the step)
    print("bench: timing the parity configurations", file=sys.stderr, flush=True)
    parity_configs = run_parity_configs(torch, pk, wl)

    per_op = []
    for i, op in enumerate(ops):
        each = sorted(light.elapsed_ms(ev[s][i], ev[s][i + 1]) for s in range(args.steps))
        ms = sum(each) / args.steps
        tflops = op.flops / (ms * 1e-3) / 1e12
        per_op.append({"op": op.name, "config": op.config, "ms": round(ms, 4),
                       "ms_median": round(each[len(each) // 2], 4), "ms_min": round(each[0], 4),
                       "tflops": round(tflops, 2), "frac_mfma_peak": round(tflops / FP32_MFMA_PEAK_TFLOPS, 4),
                       "gbs": round(op.bytes / (ms * 1e-3) / 1e9, 1)})
    dom = max(range(len(ops)), key=lambda i: per_op[i]["ms"])
    d = per_op[dom]
    roofline = {"bound": "mfma", "achieved": d["tflops"], "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(d["tflops"] / FP32_MFMA_PEAK_TFLOPS, 4),
                "traffic": measured_traffic(d["op"], d["config"]),
                "kernel": d["config"], "workload": d["op"], "avg_launch_ms": d["ms"],
                "flops_per_launch": ops[dom].flops,
                "timing": "fence-free HIP events around each launch on its stream, inside the step"}
    light.close()

    cpu = None
    if args.cpu_seconds > 0:
        import oracle
        print("bench: timing the CPU oracle sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(oracle, host, ops, args.cpu_seconds, np)

    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "ms_per_step_with_op_events": round(ms_per_step_with_op_events, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "gemm 4096^3 NN/TN/NT beta=0.5 + vgg16 conv{1..5}_1 b32 + "
                               "resnet50 bottleneck convs b32 (13 ops per step)",
                   "frac_mfma_peak": round(value / 1e3 / FP32_MFMA_PEAK_TFLOPS, 4),
                   "step_gflop": round(step_flops / 1e9, 3)},
        "roofline": roofline,
        "measured_probes": measured,
        "cpu_baseline": cpu,
        "per_op": per_op,
        "parity_configs": parity_configs,
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
