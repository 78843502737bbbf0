"""Benchmark of the ASP W4A4 + rank-32 linear layer on one MI355X.

Workload: the video-DiT FFN up-projection, M = 4096 tokens, K = 3072,
N = 14336, rank r = 32, group 64, bf16 in / out, seeded synthetic inputs
(activations N(0,1) with 1% of channels scaled by a log-uniform factor in
[10, 50]; weights N(0, 1/K); factors from the top-32 eigenvectors of a seeded
SPD Gramian).  One step = one pass of the layer's hot path over one batch:
the fused activation kernel (smoothing, group-64 INT4 quantization, packing,
down-projection) and the W4A4 GEMM (exact integer group partials on the FP6
matrix cores) with the fused bf16 branch.  The weights
are packed once before timing (they are quantized offline); every input is
resident in HBM when the timed region starts.

To keep the 256 MB Infinity Cache from serving "HBM" traffic, the steps cycle
through `--rotate` distinct copies of every input and output buffer.

Prints ONE JSON line (metric, value = effective TOPS = 2 M K N / step time,
roofline of the dominant kernel, CPU-oracle baseline).

Counter support (HBM traffic of the GEMM, scaled by a plain copy of known size):
  python bench.py --no-cpu-baseline --steps 20 --warmup 2 --copy-probe 256
      under `rocprofv3 --pmc FETCH_SIZE` and, separately, `--pmc WRITE_SIZE`
      (the copy probe runs after the timed region);
  python bench.py --reduce-counters FETCH.csv WRITE.csv
      turns the two counter-collection CSVs into profiles/traffic_asp_gemm_ffn_up.json.

Secondary measurement (not the headline line):
  python bench.py --deflated
      the same layer and line format with the paper's activation deflation
      (Eq. 8 / Eq. 9: the 4-bit path quantizes x~ - L1 t), i.e. with
      qwam_quantize_act_deflated as the activation kernel; its roofline is the
      FP64 + FP32 matrix-core work of t and of the r rank-1 updates.
  python bench.py --group 32 [--rotated] [--deflated]
      the same layer with App. B.1's group size of 32 (one float32 scale per 32
      channels, two integer partials per 64-channel MFMA); with --rotated
      --deflated this is the paper's full deployed setting.
  python bench.py --rotated [--deflated]
      the same layer with the block Hadamard rotation of Eq. 3 (B = 1024,
      applied online to the activation by the fast Walsh-Hadamard transform;
      the weights rotated offline), optionally with deflation as well: the
      paper's full deployed layer (smoothing, rotation, protected subspace).
  python bench.py --aog
      the AOG accumulation (Sec. 4.1, probe estimator): A [4096][4096] float32
      += gT gT^T for a batch of 4096 bf16 probe VJPs, the SYRK on the bf16
      matrix cores; one JSON line with its roofline and the oracle beside it.
  python bench.py --small-m
      the action-expert layers (M in {16, 32, 64}, K = 1024, N in {4096, 1024},
      r = 16): per-call latency of both kernels and algorithmic HBM GB/s, one
      JSON line per shape, rotating through enough distinct layers that the
      weights come from HBM.
  python bench.py --denoise-step
      one denoising step of a 30-block transformer (hidden 3072, FFN 14336,
      8192 tokens; per block QKV, out-projection, FFN up, FFN down, r = 32),
      every layer with its own weights and a fresh activation: aggregate
      effective TOPS, one JSON line.
"""

from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

M, K, N, R_RANK, GROUP = 4096, 3072, 14336, 32, 64
# the video-DiT layer shapes (M tokens, K in, N out); the headline line is the FFN up-projection
WORKLOADS = {"video_dit_ffn_up": (4096, 3072, 14336), "video_dit_qkv": (4096, 3072, 9216),
             "video_dit_ffn_down": (4096, 14336, 3072)}
G = K // GROUP
MFMA_PEAK = 5000.0             # MI355X dense FP8 (= dense INT8) matrix peak, TFLOP/s (TOP/s)
FP6_MFMA_PEAK = 10100.0        # MI355X dense FP6 / FP4 matrix peak, TFLOP/s: the GEMM's own dtype
BF16_MFMA_PEAK = 2500.0        # MI355X dense bf16 matrix peak, TFLOP/s
FP64_MFMA_PEAK = 78.6          # MI355X dense FP64 matrix peak, TFLOP/s
FP32_MFMA_PEAK = 157.3         # MI355X dense FP32 matrix peak, TFLOP/s
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
METRIC = "ASP W4A4+r32 linear: effective TOPS & % int8 MFMA peak at 4096×3072×14336"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_asp_gemm_ffn_up.json")
GEMM_SRCS = [os.path.join(ROOT, "paper_2609_33269_amd", "csrc", f) for f in ("qwam_gemm.hip", "qwam_device.h", "qwam_mfma.h")]
GEMM_KERNEL = "asp_gemm_kernel<32, false, 64>"
COPY_KERNEL = "(anonymous namespace)::copy_kernel("   # the streaming copy of qwam_probe_copy


def gemm_issue_ceiling(group: int = GROUP) -> float:
    """Share of the FP6 peak the GEMM's instruction mix allows with perfect overlap.

    Per wave and 64-channel span (a 64 x 64 block of y): 4 FP6 MFMAs of 32 cycles
    each per scale group (the useful work: 128 cycles at group 64), 2 bf16
    outer-product MFMAs of 64 cycles each per scale group, one FMA per output and
    scale group (64 per lane) plus 4 instructions per scale group for the bf16
    split of the token scale (the weight scale's pieces come from the pack) and
    32 unpack instructions on the VALU, 4 cycles each for a 64-wide wave.
    """
    ns = 64 // group
    mfma = ns * (4 * 32 + 2 * 64)
    valu = 4 * (ns * (64 + 4) + 32)
    return 128 / max(mfma, valu)


def algorithmic_bytes(group: int = GROUP):
    G = K // group
    act = M * K * 2 + K * 4 + R_RANK * K * 2 + M * K // 2 + M * G * 4 + M * R_RANK * 2
    gemm = M * K // 2 + M * G * 4 + M * R_RANK * 2 + N * K // 2 + N * G * 4 + N * R_RANK * 2 + M * N * 2
    return act, gemm


def source_hash(paths) -> str:
    h = hashlib.sha256()
    for path in paths:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per GEMM launch from committed rocprofv3 counters, or None if
    the kernel source changed since they were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("gemm_source_sha256_16") != source_hash(GEMM_SRCS):
        return None
    return rec.get("bytes_per_launch")


def _counter_rows(path):
    """(kernel name, value) of every dispatch in a rocprofv3 counter-collection CSV."""
    with open(path, newline="") as f:
        return [(r["Kernel_Name"], float(r["Counter_Value"])) for r in csv.DictReader(f)]


def reduce_counters(fetch_csv: str, write_csv: str, copy_mib: int):
    """HBM bytes per GEMM launch: FETCH_SIZE + WRITE_SIZE (KiB per dispatch),
    each scaled by the factor that maps the same counter of the copy probe onto
    its known byte count."""
    out = {"gemm_source_sha256_16": source_hash(GEMM_SRCS), "copy_bytes": copy_mib << 20}
    for key, path in (("fetch", fetch_csv), ("write", write_csv)):
        rows = _counter_rows(path)
        gemm = [v for k, v in rows if GEMM_KERNEL in k]
        copy = [v for k, v in rows if k.startswith(COPY_KERNEL)]
        if not gemm or not copy:
            raise SystemExit(f"{path}: no {GEMM_KERNEL} or {COPY_KERNEL} dispatches")
        g_kib, c_kib = float(np.mean(gemm)), float(np.mean(copy))
        factor = (copy_mib << 20) / (c_kib * 1024.0)
        out.update({f"{key}_kib_per_launch": round(g_kib, 1), f"copy_{key}_kib": round(c_kib, 1),
                    f"{key}_factor": round(factor, 5), f"{key}_launches": len(gemm)})
    out["bytes_per_launch"] = int(round((out["fetch_kib_per_launch"] * out["fetch_factor"] +
                                         out["write_kib_per_launch"] * out["write_factor"]) * 1024))
    out["algorithmic_bytes"] = algorithmic_bytes()[1]
    return out


def settle_clocks(step, min_seconds: float, window: int = 10, max_seconds: float = 8.0):
    """Run `step` in windows of `window` calls until at least `min_seconds`
    have passed and the last three windows agree within 2% (or `max_seconds`)."""
    import torch
    stream = torch.cuda.current_stream()
    times, n, t0 = [], 0, time.perf_counter()
    while True:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(window):
            step(n)
            n += 1
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) * 1e3 / window)
        elapsed = time.perf_counter() - t0
        last = times[-3:]
        stable = len(last) == 3 and max(last) <= 1.02 * min(last)
        if (elapsed >= min_seconds and stable) or elapsed >= max_seconds:
            return {"steps": n, "seconds": round(elapsed, 2), "stable": stable,
                    "window_us": [round(v, 1) for v in last]}


def capture_graphs(fn, n: int):
    """One CUDA/HIP graph per index i < n, each holding fn(i)."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(n):
            fn(i)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graphs = []
    for i in range(n):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn(i)
        graphs.append(g)
    for g in graphs:
        g.replay()
    torch.cuda.synchronize()
    return graphs


def graph_floor_us(n: int = 200, replays: int = 10) -> float:
    """Per-launch time of an empty kernel inside a HIP graph of n launches."""
    import torch
    from paper_2609_33269_amd import qwam
    g = capture_graphs(lambda i: [qwam.probe_empty() for _ in range(n)], 1)[0]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(replays):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / (n * replays)


def measured_peaks(sweep: bool = False):
    """What the chip sustains in plain loops (the probes of qwam_probe.h): each
    matrix-core format, the float32 VALU at 1, 2 and 4 waves per SIMD, a
    streaming copy of 2 x 1 GiB; best of three launches each."""
    import torch
    from paper_2609_33269_amd import qwam
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()

    def best_ms(launch, reps=3):
        best = None
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            launch()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1)
            best = ms if best is None else min(best, ms)
        return best

    wgs = 1024                    # 4 waves per SIMD on 256 CUs
    out = torch.empty(wgs * 256, device=dev, dtype=torch.float32)
    mfma = {}
    for kind, iters in (("fp6", 4096), ("fp4", 4096), ("fp8", 2048), ("i8", 2048), ("bf16", 2048),
                        ("bf16_2b", 1024)):
        ops = qwam.probe_mfma(kind, wgs, iters, out)
        ms = best_ms(lambda: qwam.probe_mfma(kind, wgs, iters, out))
        mfma[kind] = round(ops / (ms * 1e-3) / 1e12, 1)
    valu = {}
    for wps in (1, 2, 4):
        ow = torch.empty(256 * wps * 256, device=dev, dtype=torch.float32)
        fl = qwam.probe_valu_fma(256 * wps, 512, ow)
        ms = best_ms(lambda: qwam.probe_valu_fma(256 * wps, 512, ow))
        valu[f"{wps}_waves_per_simd"] = round(fl / (ms * 1e-3) / 1e12, 1)
    src = torch.ones((1 << 30) // 4, device=dev, dtype=torch.float32)
    dst = torch.empty_like(src)
    moved = qwam.probe_copy(src, dst)
    ms = best_ms(lambda: qwam.probe_copy(src, dst))
    copy_gbs = round(moved / (ms * 1e-3) / 1e9, 1)
    del src, dst
    torch.cuda.empty_cache()
    out = {"mfma_TOPS": mfma, "valu_fp32_fma_TFLOPs": valu, "copy_GBs": copy_gbs,
           "launch_floor_graph_us": round(graph_floor_us(), 2),
           "method": "probe loops of include/qwam_probe.h, best of 3 launches; MFMA and copy at 4 waves/SIMD"}
    if sweep:
        # the copy at smaller sizes: the bandwidth a kernel of that size can see
        # when launched back to back (as the layer's kernels are), each size
        # cycling through distinct sources and destinations that together exceed
        # the 256 MB Infinity Cache; events only at the two ends of the launches
        rows = {}
        for mib in (4, 8, 16, 32, 64, 128, 256, 512):
            n = (mib << 20) // 4
            nb = max(2, 768 // mib)
            srcs = [torch.ones(n, device=dev, dtype=torch.float32) for _ in range(nb)]
            dsts = [torch.empty(n, device=dev, dtype=torch.float32) for _ in range(nb)]
            launches = max(20, nb)
            for i in range(nb):
                qwam.probe_copy(srcs[i], dsts[i])
            best = None
            for _ in range(3):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for i in range(launches):
                    qwam.probe_copy(srcs[i % nb], dsts[(i + 1) % nb])
                e1.record(stream)
                torch.cuda.synchronize()
                ms = e0.elapsed_time(e1) / launches
                best = ms if best is None else min(best, ms)
            rows[f"{mib}MiB"] = {"us": round(best * 1e3, 2), "GBs": round(2 * (mib << 20) / (best * 1e-3) / 1e9, 1)}
            del srcs, dsts
            torch.cuda.empty_cache()
        out["copy_sweep_read_plus_write"] = rows
        out["copy_sweep_method"] = ("back-to-back launches over distinct buffers (more than the Infinity Cache), "
                                    "events at the two ends, best of 3")
    return out


def small_m_report(args):
    """Per-call latency and algorithmic HBM bandwidth of the action-expert layers.

    Latency is measured as the paper measures it, on graph replays: one HIP
    graph holds one call (both kernels) on each of `distinct_layers` packed
    layers, so every replay streams every layer's weights from HBM (together
    they exceed the 256 MB Infinity Cache)."""
    import torch
    from paper_2609_33269_amd import calib, inputs, qwam

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def graph_us(fn, n, replays=10):
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for i in range(n):
                fn(i)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(n):
                fn(i)
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(replays):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / (replays * n)

    # floor: a graph of one-element kernels
    one = torch.zeros(1, device=dev)
    floor_us = graph_us(lambda i: one.add_(1.0), 512)

    Ka, ra, Ga = 1024, 16, 1024 // GROUP
    for (Ms, Ns) in inputs.ACTION_EXPERT_SHAPES:
        d = inputs.action_expert(Ms, Ns)
        x0 = torch.from_numpy(d.x.view(np.int16)).view(torch.bfloat16).to(dev)
        w0 = torch.from_numpy(d.w.view(np.int16)).view(torch.bfloat16).to(dev)
        f = calib.build_layer(x0, w0, calib.protected_basis(torch.from_numpy(d.a), ra))
        L0 = qwam.make_layer(f["R"], f["lam"], f["L1"], f["L2"])
        del f, w0
        wbytes = Ns * Ka // 2 + Ns * Ga * 4 + Ns * ra * 2 + Ka * 4 + ra * Ka * 2
        nrot = int(min(1024, max(2, (768 << 20) // wbytes)))        # > the 256 MB Infinity Cache
        layers = [L0] + [qwam.PackedLayer(K=Ka, N=Ns, r=ra, wq=L0.wq.clone(), ws=L0.ws.clone(), wsp=L0.wsp.clone(),
                                          inv_smooth=L0.inv_smooth.clone(), L1t=L0.L1t.clone(),
                                          L2t=L0.L2t.clone(), L1=L0.L1.clone(), L1f=L0.L1f.clone()) for _ in range(nrot - 1)]
        xq = torch.empty((Ms, Ka // 2), dtype=torch.uint8, device=dev)
        xs = torch.empty((Ga, Ms), dtype=torch.float32, device=dev)
        t = torch.empty((Ms, ra), dtype=torch.bfloat16, device=dev)
        y = torch.empty((Ms, Ns), dtype=torch.bfloat16, device=dev)

        def call(i):
            L = layers[i]
            qwam.quantize_act(L, x0, out=(xq, xs, t))
            qwam.asp_linear(L, xq, xs, t, out=y)

        us = graph_us(call, nrot)
        us_fused = graph_us(lambda i: qwam.asp_layer(layers[i], x0, out=y), nrot)
        # App. B.1's full setting (group 32, Hadamard rotation, deflation) on
        # the same shape: the two-call path (the fused layer takes group 64
        # without rotation only)
        w0 = torch.from_numpy(d.w.view(np.int16)).view(torch.bfloat16).to(dev)
        fp = calib.build_layer(x0, w0, calib.protected_basis(torch.from_numpy(d.a), ra), hadamard=True)
        Lp = qwam.make_layer(fp["R"], fp["lam"], fp["L1"], fp["L2"], hadamard=fp["hadamard"], group=32)
        del fp, w0
        players = [Lp] + [qwam.PackedLayer(K=Ka, N=Ns, r=ra, wq=Lp.wq.clone(), ws=Lp.ws.clone(), wsp=Lp.wsp.clone(),
                                           inv_smooth=Lp.inv_smooth.clone(), L1t=Lp.L1t.clone(),
                                           L2t=Lp.L2t.clone(), L1=Lp.L1.clone(), L1f=Lp.L1f.clone(), hadamard=Lp.hadamard,
                                           group=32) for _ in range(nrot - 1)]
        xs32 = torch.empty((Ka // 32, Ms), dtype=torch.float32, device=dev)

        def call_paper(i):
            L = players[i]
            qwam.quantize_act_deflated(L, x0, out=(xq, xs32, t))
            qwam.asp_linear(L, xq, xs32, t, out=y)

        us_paper = graph_us(call_paper, nrot)
        us_paper_act = graph_us(lambda i: qwam.quantize_act_deflated(players[i], x0, out=(xq, xs32, t)), nrot)
        us_paper_gemm = graph_us(lambda i: qwam.asp_linear(players[i], xq, xs32, t, out=y), nrot)
        del players, Lp
        us1 = graph_us(lambda i: qwam.quantize_act(layers[i], x0, out=(xq, xs, t)), nrot)
        us2 = graph_us(lambda i: qwam.asp_linear(layers[i], xq, xs, t, out=y), nrot)
        # the bf16 linear it replaces (hipBLASLt through torch), same graph method,
        # as many distinct bf16 weights as fit the same rotation bytes
        nb = int(min(nrot, max(2, (768 << 20) // (Ns * Ka * 2))))
        wbf = [torch.randn((Ns, Ka), device=dev, dtype=torch.bfloat16) for _ in range(nb)]
        ybf = torch.empty((Ms, Ns), device=dev, dtype=torch.bfloat16)
        us_bf16 = graph_us(lambda i: torch.matmul(x0, wbf[i].t(), out=ybf), nb)
        del wbf
        b1 = Ms * Ka * 2 + Ka * 4 + ra * Ka * 2 + Ms * Ka // 2 + Ms * Ga * 4 + Ms * ra * 2
        b2 = (Ms * Ka // 2 + Ms * Ga * 4 + Ms * ra * 2 + Ns * Ka // 2 + Ns * Ga * 4 + Ns * ra * 2
              + Ms * Ns * 2)
        print(json.dumps({
            "workload": "action_expert", "M": Ms, "K": Ka, "N": Ns, "r": ra,
            "us_per_call": round(us, 2), "us_quantize_act": round(us1, 2), "us_asp_gemm": round(us2, 2),
            "us_fused_layer": round(us_fused, 2), "fused_GBs": round((b1 + b2) / (us_fused * 1e-6) / 1e9, 1),
            "us_group32_rotated_deflated_two_call": round(us_paper, 2),
            "us_group32_rotated_deflated_act": round(us_paper_act, 2),
            "us_group32_gemm": round(us_paper_gemm, 2),
            "fused_speedup_vs_bf16_linear": round(us_bf16 / us_fused, 3),
            "algorithmic_bytes": b1 + b2, "GBs": round((b1 + b2) / (us * 1e-6) / 1e9, 1),
            "gemm_GBs": round(b2 / (us2 * 1e-6) / 1e9, 1),
            "hbm_frac": round((b1 + b2) / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "bf16_linear_us": round(us_bf16, 2), "speedup_vs_bf16_linear": round(us_bf16 / us, 3),
            "graph_kernel_floor_us": round(floor_us, 2), "distinct_layers": nrot,
            "timing": "HIP graph replay", "data": "synthetic"}), flush=True)
        del layers, L0, x0
        torch.cuda.empty_cache()


def denoise_step_report(args):
    """Aggregate throughput of the 120 ASP layers of one denoising step.

    The weights and activations of 120 full-size layers are drawn on the GPU
    (seeded torch generators) from the same recipes as the seeded inputs
    module: W ~ N(0, 1/K); x ~ N(0, 1) with 1% of channels scaled by a
    log-uniform factor in [10, 50]; the FFN down-projection gets bf16(GELU(z)),
    z ~ N(0, 1).  Each layer is calibrated (smoothing, top-32 eigenvectors of a
    seeded stand-in Gramian, L1 / L2, R) and packed by the library, as offline.
    """
    import math
    import torch
    from paper_2609_33269_amd import calib, inputs, qwam

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    Ms, rr = 8192, 32
    layers, acts, flops = [], [], 0
    t0 = time.perf_counter()
    for b in range(inputs.DENOISE_BLOCKS):
        for which, (name, Ks, Ns) in enumerate(inputs.DENOISE_BLOCK):
            gen = torch.Generator(device=dev)
            gen.manual_seed(4_000_000 + 4 * b + which)
            w = (torch.randn((Ns, Ks), generator=gen, device=dev) / math.sqrt(Ks)).to(torch.bfloat16)
            z = torch.randn((Ms, Ks), generator=gen, device=dev)
            if name == "ffn_down":
                x = torch.nn.functional.gelu(z).to(torch.bfloat16)
            else:
                n_out = max(1, Ks // 100)
                cols = torch.randperm(Ks, generator=gen, device=dev)[:n_out]
                fac = torch.exp(torch.empty(n_out, device=dev).uniform_(math.log(10.0), math.log(50.0),
                                                                         generator=gen))
                z[:, cols] *= fac
                x = z.to(torch.bfloat16)
            del z
            a = torch.randn((Ks, 64), generator=gen, device=dev, dtype=torch.float64)
            f = calib.build_layer(x, w, calib.protected_basis(a, rr))
            layers.append(qwam.make_layer(f["R"], f["lam"], f["L1"], f["L2"]))
            acts.append(x)
            flops += 2.0 * Ms * Ks * Ns
            del f, w, a
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t0
    print(f"[bench] {len(layers)} layers drawn, calibrated and packed in {setup_s:.1f} s", file=sys.stderr,
          flush=True)

    bufs = {}
    for L in layers:
        if (L.K, L.N) not in bufs:
            bufs[(L.K, L.N)] = (torch.empty((Ms, L.K // 2), dtype=torch.uint8, device=dev),
                                torch.empty((L.K // GROUP, Ms), dtype=torch.float32, device=dev),
                                torch.empty((Ms, rr), dtype=torch.bfloat16, device=dev),
                                torch.empty((Ms, L.N), dtype=torch.bfloat16, device=dev))

    def step():
        for L, x in zip(layers, acts):
            xq, xs, t, y = bufs[(L.K, L.N)]
            qwam.quantize_act(L, x, out=(xq, xs, t))
            qwam.asp_linear(L, xq, xs, t, out=y)

    stream = torch.cuda.current_stream()
    # warm up by time (clocks settle), then the median of 5 steps, each
    # bracketed by its own events
    settle = settle_clocks(lambda _: step(), min_seconds=1.0, window=1, max_seconds=6.0)
    steps = 5
    per = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        step()
        e1.record(stream)
        torch.cuda.synchronize()
        per.append(e0.elapsed_time(e1))
    ms = float(np.median(per))
    print(json.dumps({
        "workload": "denoise_step", "blocks": inputs.DENOISE_BLOCKS, "layers": len(layers), "M": Ms, "r": rr,
        "layer_shapes": [[n, k, nn] for n, k, nn in inputs.DENOISE_BLOCK],
        "ms_per_step": round(ms, 3), "effective_TOPS": round(flops / (ms * 1e-3) / 1e12, 1),
        "frac_of_5P_peak": round(flops / (ms * 1e-3) / 1e12 / MFMA_PEAK, 4), "steps": steps,
        "timing": "median of 5 steps, each between two events, after a time-based warm-up",
        "step_ms": [round(v, 3) for v in per], "clock_settle": settle,
        "dense_equivalent_ops": flops, "data": "synthetic, drawn on the GPU"}), flush=True)


def deflated_act_roofline(k1_ms: float):
    """Matrix-core work of the deflated activation kernel: t in double
    (2 M K r flops at the FP64 peak) and the r rank-1 updates in float
    (2 M K r flops at the FP32 peak).  `peak` is the rate at which both
    together would take their ideal time."""
    flops = 2.0 * M * K * R_RANK
    ideal_s = flops / (FP64_MFMA_PEAK * 1e12) + flops / (FP32_MFMA_PEAK * 1e12)
    peak = 2.0 * flops / ideal_s / 1e12
    achieved = 2.0 * flops / (k1_ms * 1e-3) / 1e12
    return {"bound": "mfma (fp64 t + fp32 rank-1 updates)", "achieved": round(achieved, 2),
            "peak": round(peak, 2), "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
            "ideal_us": round(ideal_s * 1e6, 2), "flops": 2.0 * flops}


def aog_report(args):
    """AOG accumulation A += gT gT^T (d = 4096, n = 4096 per call), rotating
    through distinct gT batches and accumulators so that the 256 MB Infinity
    Cache does not hold them; the CPU oracle timed on a row sample."""
    import torch
    from paper_2609_33269_amd import qwam

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    d, n, nrot = 4096, 4096, 6
    gen = torch.Generator(device=dev)
    gen.manual_seed(5_000_000)
    col = torch.exp(-torch.arange(d, device=dev, dtype=torch.float32) / (d / 8.0))
    gts = [(torch.randn((d, n), generator=gen, device=dev) * col[torch.randperm(d, generator=gen, device=dev)][:, None])
           .to(torch.bfloat16) for _ in range(nrot)]
    accs = [torch.zeros((d, d), dtype=torch.float32, device=dev) for _ in range(nrot)]
    stream = torch.cuda.current_stream()
    for i in range(args.warmup):
        qwam.aog_accumulate(gts[i % nrot], accs[i % nrot])
    torch.cuda.synchronize()
    steps = args.steps
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(steps):
        qwam.aog_accumulate(gts[i % nrot], accs[i % nrot])
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / steps
    flops = float(n) * d * (d + 1)               # the symmetric rank-n update
    bytes_ = d * n * 2 + 2 * d * d * 4            # gT once, A read and written once
    tflops = flops / (us * 1e-6) / 1e12
    # the eigensolve that follows the last batch: top-32 eigenvectors of
    # G~ = H diag(lam) (A / (N P)) diag(lam) H (B = 1024), 10 products with G~;
    # each product reads A once (HBM-bound), so its roofline is HBM
    r_eig, iters = 32, 10
    lam = torch.exp(torch.empty(d, device=dev).uniform_(-1.0, 1.0, generator=gen))
    ws = torch.empty(qwam.aog_protected_basis_workspace(d, r_eig), dtype=torch.uint8, device=dev)
    for i in range(2):
        qwam.aog_protected_basis(accs[i], r_eig, iters=iters, scale=1.0 / n, lam=lam, hadamard=1024, workspace=ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(5):
        qwam.aog_protected_basis(accs[i % nrot], r_eig, iters=iters, scale=1.0 / n, lam=lam, hadamard=1024,
                                 workspace=ws)
    e1.record(stream)
    torch.cuda.synchronize()
    eig_us = e0.elapsed_time(e1) * 1e3 / 5
    eig_bytes = (iters + 1) * d * d * 4
    # the CPU oracle (float64 rank-k update) on column samples of the same batch
    print("[bench] oracle accumulation (host)", file=sys.stderr, flush=True)
    from oracle import qwam_oracle as O
    g_bits = gts[0].view(torch.int16).cpu().numpy().view(np.uint16)
    cols = 256
    A_cpu = np.zeros((d, d))
    t0 = time.perf_counter()
    reps = 0
    while reps == 0 or time.perf_counter() - t0 < min(args.cpu_seconds, 10.0):
        A_cpu = O.aog_accumulate(A_cpu, g_bits[:, (reps * cols) % n:(reps * cols) % n + cols])
        reps += 1
    dt = time.perf_counter() - t0
    cpu_tflops = float(cols) * d * (d + 1) * reps / dt / 1e12
    # the oracle's eigensolve (numpy eigh in float64), one call on the smoothed
    # estimate diag(lam) G^ diag(lam); the oracle's dense block rotation of a
    # 4096 x 4096 matrix alone takes minutes on the host, so the sample leaves it out
    eig_cpu = None
    if not args.no_cpu_baseline:
        print("[bench] oracle eigensolve (host, one call)", file=sys.stderr, flush=True)
        Gt = O.rotated_aog(O.aog_estimate(accs[0].double().cpu().numpy(), n, 1), lam.double().cpu().numpy(), 0)
        t0 = time.perf_counter()
        O.protected_basis_eigh(Gt, r_eig)
        eig_cpu = {"seconds": round(time.perf_counter() - t0, 2), "kind": "oracle (numpy eigh, float64)",
                   "cores": os.cpu_count(), "sample": f"one call at d = {d}, smoothed estimate without the rotation"}
        del Gt
    print(json.dumps({
        "metric": "AOG accumulation A += gT gT^T: TFLOP/s", "value": round(tflops, 1), "unit": "TFLOP/s",
        "n_gpus": 1, "steps": steps, "warmup": args.warmup, "ms_per_step": round(us / 1e3, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16 products (exact), f32 accumulate", "data": "synthetic",
        "config": {"workload": "aog_accumulate", "d": d, "n": n, "rotated_buffer_sets": nrot},
        "roofline": {"bound": "mfma", "kernel": "aog_syrk_kernel", "achieved": round(tflops, 1),
                     "peak": BF16_MFMA_PEAK, "unit": "TFLOP/s", "frac": round(tflops / BF16_MFMA_PEAK, 4),
                     "traffic": None, "algorithmic_bytes": bytes_,
                     "hbm_GBs": round(bytes_ / (us * 1e-6) / 1e9, 1)},
        "eigensolve": {"kernel": "qwam_aog_protected_basis", "d": d, "r": r_eig, "iters": iters, "block": 64,
                       "hadamard": 1024, "us": round(eig_us, 1),
                       "A_bytes_read": eig_bytes, "hbm_GBs": round(eig_bytes / (eig_us * 1e-6) / 1e9, 1),
                       "frac_of_hbm_peak": round(eig_bytes / (eig_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                       "cpu_oracle": eig_cpu},
        "cpu_baseline": {"value": round(cpu_tflops, 5), "unit": "TFLOP/s", "cores": os.cpu_count(), "kind": "oracle",
                         "sample": f"{reps} calls of the oracle on {cols} of the {n} VJPs (all {d} channels) in "
                                   f"{dt:.1f} s; value = cols*d*(d+1)*calls/time"}}), flush=True)


def cpu_baseline(draws, seconds: float = 12.0, deflate: bool = False, rotate: bool = False, group: int = GROUP):
    """The CPU oracle as it stands, timed on a bounded token sample of the same
    layer (weights packed beforehand, as on the GPU)."""
    from oracle import qwam_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:   # pragma: no cover
        threads = 1
    V = O.protected_basis_from_factor(draws.a, R_RANK)
    f = O.build_layer(draws.x, draws.w, V, hadamard=rotate)
    # the weight codes and scales (the packed bytes themselves are not needed here)
    qw, sw = O.quantize_groups(f["R"], group)
    inv_lam = O.inverse_smoothing(f["lam"])
    chunk = 32
    done = 0
    t0 = time.perf_counter()
    while done + chunk <= M:
        rows = slice(done, done + chunk)
        quant = O.quantize_activations_deflated if deflate else O.quantize_activations
        xq, sx, t, qx, _ = quant(draws.x[rows], inv_lam, f["L1"], f["hadamard"], group)
        P = O.group_partials(qx, qw, group)
        O.asp_output(sx, sw, P, t, f["L2"])
        done += chunk
        if time.perf_counter() - t0 >= seconds:
            break
    dt = time.perf_counter() - t0
    return {"value": 2.0 * done * K * N / dt / 1e12, "unit": "TOPS", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{done} of {M} tokens (chunks of {chunk}) of the {M}x{K}x{N} r{R_RANK} layer"
                      f"{' with rotation' if rotate else ''}{' with deflation' if deflate else ''}"
                      f"{', group 32' if group == 32 else ''}, "
                      f"weights packed beforehand; {dt:.1f} s; value = 2*tokens*K*N/time"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--settle", type=float, default=1.5,
                    help="seconds of clock-settling steps before the warmup steps (always run)")
    ap.add_argument("--no-peaks", action="store_true", help="skip the measured-peak probes")
    ap.add_argument("--rotate", type=int, default=24, help="distinct buffer sets cycled through")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="after timing, run a plain float32 copy kernel over MIB MiB five times")
    ap.add_argument("--reduce-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"))
    ap.add_argument("--copy-mib", type=int, default=256, help="copy-probe size the counters were taken with")
    ap.add_argument("--deflated", action="store_true",
                    help="the same layer with the deflated activation kernel (Eq. 8 / Eq. 9)")
    ap.add_argument("--group", type=int, default=GROUP, choices=(32, 64),
                    help="channels per quantization scale (64, or the paper's 32)")
    ap.add_argument("--rotated", action="store_true",
                    help="the same layer with the block Hadamard rotation (Eq. 3) on both operands")
    ap.add_argument("--workload", default="video_dit_ffn_up", choices=sorted(WORKLOADS),
                    help="layer shape of the line (the metric is quoted on video_dit_ffn_up)")
    ap.add_argument("--aog", action="store_true", help="report the AOG accumulation kernel instead")
    ap.add_argument("--peaks", action="store_true",
                    help="print the measured chip peaks (MFMA loops, VALU, copy and a copy-size sweep) instead")
    ap.add_argument("--small-m", action="store_true", help="report the action-expert layers instead")
    ap.add_argument("--denoise-step", action="store_true", help="report one 120-layer denoising step instead")
    args = ap.parse_args()
    if args.reduce_counters:
        rec = reduce_counters(*args.reduce_counters, args.copy_mib)
        os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
        with open(TRAFFIC_FILE, "w") as f:
            json.dump(rec, f, indent=1)
            f.write("\n")
        print(json.dumps(rec))
        return
    global M, K, N, G
    M, K, N = WORKLOADS[args.workload]
    G = K // GROUP
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the ASP layer is "
              f"implemented and measured on a single GPU, with no sharding", file=sys.stderr)
        sys.exit(2)

    if args.peaks:
        import torch
        torch.cuda.set_device(0)
        print(json.dumps({"measured_peaks": measured_peaks(sweep=True)}), flush=True)
        return
    if args.aog:
        aog_report(args)
        return
    if args.small_m:
        small_m_report(args)
        return
    if args.denoise_step:
        denoise_step_report(args)
        return

    import torch
    from paper_2609_33269_amd import calib, inputs, qwam

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    print(f"[bench] drawing inputs {args.workload} {M}x{K}x{N} r{R_RANK}", file=sys.stderr, flush=True)
    draws = getattr(inputs, args.workload)()
    x0 = torch.from_numpy(draws.x.view(np.int16)).view(torch.bfloat16).to(dev)
    w0 = torch.from_numpy(draws.w.view(np.int16)).view(torch.bfloat16).to(dev)
    V = calib.protected_basis(torch.from_numpy(draws.a), R_RANK)
    f = calib.build_layer(x0, w0, V, hadamard=args.rotated)
    layer0 = qwam.make_layer(f["R"], f["lam"], f["L1"], f["L2"], hadamard=f["hadamard"], group=args.group)
    del f, w0
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    nrot = max(1, args.rotate)
    layers, xins, outs = [], [], []
    for i in range(nrot):
        L = layer0 if i == 0 else qwam.PackedLayer(
            K=K, N=N, r=R_RANK, wq=layer0.wq.clone(), ws=layer0.ws.clone(), wsp=layer0.wsp.clone(),
            inv_smooth=layer0.inv_smooth.clone(), L1t=layer0.L1t.clone(), L2t=layer0.L2t.clone(),
            L1=layer0.L1.clone(), L1f=layer0.L1f.clone(), hadamard=layer0.hadamard, group=layer0.group)
        layers.append(L)
        xins.append(x0 if i == 0 else x0.clone())
        outs.append((torch.empty((M, K // 2), dtype=torch.uint8, device=dev),
                     torch.empty((K // args.group, M), dtype=torch.float32, device=dev),
                     torch.empty((M, R_RANK), dtype=torch.bfloat16, device=dev),
                     torch.empty((M, N), dtype=torch.bfloat16, device=dev)))
    stream = torch.cuda.current_stream()
    act_fn = qwam.quantize_act_deflated if args.deflated else qwam.quantize_act

    def step(i):
        j = i % nrot
        xq, xs, t, y = outs[j]
        act_fn(layers[j], xins[j], out=(xq, xs, t))
        qwam.asp_linear(layers[j], xq, xs, t, out=y)

    # HIP graphs of the step (both kernels): one holding the steps of all nrot
    # buffer sets in order, and one per buffer set for a remainder; replayed
    # beside the timed region (captured first, so that the clock settle and
    # the warmup come right before the timed region)
    block = capture_graphs(lambda _: [step(j) for j in range(nrot)], 1)[0]
    singles = capture_graphs(lambda j: step(j), nrot)

    def replay_steps(n):
        for _ in range(n // nrot):
            block.replay()
        for i in range(n % nrot):
            singles[i].replay()

    # clock settle: the first calls on a fresh box run at lower clocks, so the
    # steps are warmed by time (at least `--settle` seconds, then until three
    # consecutive 10-step windows agree within 2%), whatever --warmup says
    settle = settle_clocks(step, args.settle)
    print(f"[bench] clocks settled after {settle['steps']} steps / {settle['seconds']:.2f} s "
          f"(last windows {settle['window_us']} us/step); warmup {args.warmup} steps", file=sys.stderr, flush=True)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    def launch_steps(n):
        for i in range(n):
            step(i)

    # the timed region: K steps launched back to back, no event inside
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    launch_steps(args.steps)
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_step = total_ms / args.steps

    rep_steps = max(100, args.steps)

    def timed(fn, n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn(n)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    # 10 repeats of max(100, K) steps, launched and replayed from the graphs: medians
    med_ms = float(np.median([timed(launch_steps, rep_steps) for _ in range(10)]))
    graph_ms = timed(replay_steps, args.steps)
    graph_med_ms = float(np.median([timed(replay_steps, rep_steps) for _ in range(10)]))

    # per-kernel durations: one HIP graph per kernel holding one launch on
    # each buffer set, replayed until at least `rep_steps` launches ran back to
    # back, events only at the two ends (so the mean includes the gaps between
    # consecutive launches, but no host time: a launch through the Python
    # binding costs more host time than the activation kernel takes); median
    # of 5
    def act_one(j):
        act_fn(layers[j], xins[j], out=outs[j][:3])

    def gemm_one(j):
        xq, xs, t, y = outs[j]
        qwam.asp_linear(layers[j], xq, xs, t, out=y)

    act_graph = capture_graphs(lambda _: [act_one(j) for j in range(nrot)], 1)[0]
    gemm_graph = capture_graphs(lambda _: [gemm_one(j) for j in range(nrot)], 1)[0]
    reps = max(1, -(-rep_steps // nrot))

    def replayed(g):
        def run(_n):
            for _ in range(reps):
                g.replay()
        return run

    k1_all = [timed(replayed(act_graph), reps * nrot) for _ in range(5)]
    k2_all = [timed(replayed(gemm_graph), reps * nrot) for _ in range(5)]
    k1_ms, k2_ms = float(np.median(k1_all)), float(np.median(k2_all))
    del block, singles, act_graph, gemm_graph
    print(f"[bench] {args.steps} steps: {ms_step * 1e3:.1f} us/step (median of 10 x {rep_steps}: {med_ms * 1e3:.1f}; "
          f"graph replay {graph_ms * 1e3:.1f}, median {graph_med_ms * 1e3:.1f}); act kernel {k1_ms * 1e3:.1f} us, "
          f"gemm {k2_ms * 1e3:.1f} us", file=sys.stderr, flush=True)
    floor_us = graph_floor_us()

    int_ops = 2.0 * M * K * N
    eff_tops = int_ops / (ms_step * 1e-3) / 1e12
    k2_tops = int_ops / (k2_ms * 1e-3) / 1e12
    act_bytes, gemm_bytes = algorithmic_bytes(args.group)
    k1_gbs = act_bytes / (k1_ms * 1e-3) / 1e9

    # secondary: the bf16 linear the layer replaces (hipBLASLt through torch), same shape
    wb = torch.randn((N, K), device=dev, dtype=torch.bfloat16)
    for _ in range(5):
        torch.nn.functional.linear(x0, wb)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(20):
        torch.nn.functional.linear(x0, wb)
    e1.record(stream)
    torch.cuda.synchronize()
    bf16_ms = e0.elapsed_time(e1) / 20
    del wb

    if args.copy_probe > 0:
        n = (args.copy_probe << 20) // 4
        src_t = torch.ones(n, device=dev, dtype=torch.float32)
        dst_t = torch.empty_like(src_t)
        for _ in range(5):
            qwam.probe_copy(src_t, dst_t)    # reads and writes copy_probe MiB each
        torch.cuda.synchronize()
        del src_t, dst_t
    peaks = None if args.no_peaks else measured_peaks()

    traffic = measured_traffic() if (args.group == GROUP and args.workload == "video_dit_ffn_up") else None
    act_name = ("quantize_act_rotated" if args.rotated else "quantize_act") + ("_deflated" if args.deflated else "")
    out = {
        "metric": METRIC if args.workload == "video_dit_ffn_up" else METRIC.replace("4096×3072×14336", f"{M}×{K}×{N}"),
        "value": round(eff_tops, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int4 codes as fp6-e2m3 MFMA operands (exact int partials); per-group scale products "
                 "sx*sw on bf16 MFMA from two-piece bf16 splits (~2^-15 rel); f32 accumulate; bf16 out",
        "data": "synthetic",
        "config": {"workload": args.workload + ("_rotated" if args.rotated else "")
                   + ("_deflated" if args.deflated else "") + ("_group32" if args.group == 32 else ""),
                   "M": M, "K": K, "N": N, "r": R_RANK, "group": args.group,
                   "act": ("bf16(GELU_erf(N(0,1)))" if args.workload == "video_dit_ffn_down"
                           else "N(0,1), 1% channels x U_log(10,50)"), "weights": "N(0,1/K)",
                   "rotated_buffer_sets": nrot},
        "roofline": {"bound": "mfma", "kernel": f"asp_gemm_kernel<{R_RANK}, false, {args.group}>",
                     "achieved": round(k2_tops, 1),
                     "peak": FP6_MFMA_PEAK, "unit": "TFLOP/s", "frac": round(k2_tops / FP6_MFMA_PEAK, 4),
                     "traffic": traffic, "algorithmic_bytes": gemm_bytes},
        "layer_frac_int8_peak": round(eff_tops / MFMA_PEAK, 4),
        "kernels_us": {act_name: round(k1_ms * 1e3, 2), "asp_gemm": round(k2_ms * 1e3, 2),
                       "timing": f"per launch: a HIP graph of {nrot} launches of the kernel (one per buffer set) "
                                 f"replayed {reps} times back to back between two events, median of 5"},
        "timing": {"method": f"{args.steps} steps (both kernels) launched back to back on one stream, events "
                             f"only at the two ends",
                   "repeat_median_ms_per_step": round(med_ms, 5), "repeats": f"10 x {rep_steps} steps",
                   "graph_replay_ms_per_step": round(graph_ms, 5),
                   "graph_replay_repeat_median_ms_per_step": round(graph_med_ms, 5),
                   "graph": f"HIP graphs of {nrot} steps (one per pass over the buffer sets)",
                   "clock_settle": settle, "graph_launch_floor_us": round(floor_us, 2)},
        "quantize_act_roofline": {"bound": "hbm", "achieved": round(k1_gbs, 1), "peak": HBM_PEAK_GBS,
                                  "unit": "GB/s", "frac": round(k1_gbs / HBM_PEAK_GBS, 4),
                                  "algorithmic_bytes": act_bytes},
        "gemm_issue_ceiling_frac": round(gemm_issue_ceiling(args.group), 4),
        "bf16_linear_us": round(bf16_ms * 1e3, 2),
        "speedup_vs_bf16_linear": round(bf16_ms / ms_step, 3),
    }
    if peaks is not None:
        out["measured_peaks"] = peaks
        out["roofline"]["frac_of_measured_fp6_loop"] = round(k2_tops / peaks["mfma_TOPS"]["fp6"], 4)
        out["layer_frac_measured_i8_loop"] = round(eff_tops / peaks["mfma_TOPS"]["i8"], 4)
        out["quantize_act_roofline"]["frac_of_measured_copy"] = round(k1_gbs / peaks["copy_GBs"], 4)
    if args.deflated:
        out[act_name + "_roofline"] = deflated_act_roofline(k1_ms)
    if args.rotated:
        # the transform's own work: log2(B) float32 additions per element, on the
        # non-packed VALU (16 lanes per SIMD per clock, 1024 SIMDs, 2.4 GHz)
        adds = float(M) * K * 10
        out["fwht_adds"] = adds
        out["fwht_valu_us"] = round(adds / (1024 * 16 * 2.4e9) * 1e6, 2)
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a token sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(draws, args.cpu_seconds, deflate=args.deflated, rotate=args.rotated,
                                           group=args.group)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
