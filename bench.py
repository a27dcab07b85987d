#!/usr/bin/env python3
"""Benchmark: batch-1 fp32 conv2d forward on one MI355X.

One step = one ilpm_conv2d_fwd call on the workload (default: the early
VGG-style layer, input [1,64,224,224], weights [64,64,3,3], bias, stride 1,
pad 1), with every tensor already resident in HBM.  Prints ONE JSON line.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--all]

Before the counted warm-up (--warmup) every timed layer gets an untimed
spin-up of the same launch, bounded by wall-clock time (--spinup-ms, default
300 ms; its calls and milliseconds are in the line): in a fresh process, and
after the GPU has idled while the host drew the next layer's inputs, the first
few hundred calls run slower (on the VGG-early layer, 400-call batches from
process start averaged 46, 32.1, then 31.1-31.3 us).  The timed region itself
is exactly --steps back-to-back calls.

Besides the headline layer, the line carries a compact row per other workload
("configs": the tiny layer, ResNet conv4.x, the strided layer, the 1x1 and
5x5 deep layers, and the VGG-16 stack end to end with its per-layer times):
us per call, GFLOP/s, the roofline bound and fraction, and cold us (HBM-bound
rows, each call after a 512 MiB cache scrub).

--all also times every other workload, the rest of ResNet's 3x3 layer set and
VGG-16's first layer, then the VGG-16 conv stack layer by layer, and writes the
table to --report (JSON) without changing the line.

--vgg16-stack REPS times only the VGG-16 stack end to end (for kernel traces).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("batch-1 conv2d fwd µs/layer and GFLOP/s (2·C_out·C_in·K²·H_out·W_out)"
          " + % roofline")
PEAK_FP32_TFLOPS = 157.3   # MI355X dense fp32 (matrix cores)
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def out_size(n, k, s, p):
    return (n + 2 * p - k) // s + 1


def layer_work(c_in, h, w, c_out, k, s, p, bias):
    """Nominal FLOPs (padding taps included) and compulsory bytes (input,
    weights, bias and output each moved once, fp32)."""
    ho, wo = out_size(h, k, s, p), out_size(w, k, s, p)
    flops = 2.0 * c_out * c_in * k * k * ho * wo
    nbytes = 4.0 * (c_in * h * w + c_out * c_in * k * k + (c_out if bias else 0) + c_out * ho * wo)
    return flops, nbytes, ho, wo


def roofline_floor_us(flops, nbytes):
    tc = flops / (PEAK_FP32_TFLOPS * 1e12) * 1e6
    tm = nbytes / (PEAK_HBM_GBS * 1e9) * 1e6
    return max(tc, tm), ("mfma" if tc >= tm else "hbm")


def kernel_source_digest():
    """sha256 (first 16 hex digits) of the kernel and library sources under
    csrc/, the measured plan tables (tuned_plans*.inc) left out: those choose
    among the kernels without changing any, and a traffic entry names the
    plan it was measured on."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1909_02765_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.startswith("tuned_plans") and name.endswith(".inc"):
            continue
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, digest, plan_name):
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current kernel sources and the plan that runs now; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    e = t.get(workload)
    if not e or e.get("kernel_digest") != digest or e.get("plan") != plan_name:
        return None
    return e.get("hbm_bytes_per_launch")


SPINUP = {"ms": 300.0}  # set from --spinup-ms


def spin_up(torch, launch, ms=None):
    """Untimed back-to-back calls of `launch` until `ms` milliseconds of wall
    clock have passed (checked every 50 calls, after a synchronisation), so
    that the GPU is at its steady state when the counted warm-up starts.
    Returns (calls, ms spent)."""
    ms = SPINUP["ms"] if ms is None else ms
    t0 = time.perf_counter()
    calls = 0
    while (time.perf_counter() - t0) * 1e3 < ms:
        for _ in range(50):
            launch()
        calls += 50
        torch.cuda.synchronize()
    return calls, (time.perf_counter() - t0) * 1e3


def time_layer(torch, ilpm, x, w, b, s, p, out, steps, warmup, spin=None):
    """Mean µs per call over `steps` back-to-back ilpm_conv2d_fwd calls on the
    current stream, bracketed by events recorded on that same stream (after
    the untimed spin-up and `warmup` counted warm-up calls).  `spin`, a dict,
    receives the spin-up's calls and milliseconds."""
    launch = ilpm.conv2d_launcher(x, w, b, s, p, out)
    calls, ms = spin_up(torch, launch)
    if spin is not None:
        spin.update(calls=calls, ms=round(ms, 1))
    for _ in range(warmup):
        launch()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        launch()
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) * 1000.0 / steps


def time_layer_graph(torch, ilpm, x, w, b, s, p, out, steps, per_graph=20):
    """Mean µs per call when the same calls are replayed from a captured HIP
    graph of `per_graph` launches (no host launch cost between calls).  The
    library allocates nothing during capture: the calls made before it have
    already sized its workspace."""
    return time_graph(torch, lambda: ilpm.conv2d_launcher(x, w, b, s, p, out), steps, per_graph)


def time_graph(torch, make_launch, steps, per_graph=20):
    """time_layer_graph for any launcher: make_launch() is called with the
    capture stream current, so the launcher it returns is bound to it."""
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        launch = make_launch()
        for _ in range(3):
            launch()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for _ in range(per_graph):
                launch()
    torch.cuda.synchronize()
    reps = max(1, steps // per_graph)
    spin_up(torch, g.replay)
    for _ in range(max(1, reps // 10)):
        g.replay()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(reps):
        g.replay()
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) * 1000.0 / (reps * per_graph)


def time_prepacked(torch, ilpm, x, w, b, s, p, out, plan, steps, warmup):
    """Mean µs per call of the same plan on weights packed beforehand
    (ilpm_conv2d_prepack_weights, once, outside the timed calls)."""
    c_out, _, k, _ = w.shape
    packed = ilpm.prepack_weights(w, plan)
    launch = ilpm.conv2d_prepacked_launcher(x, packed, c_out, k, b, s, p, out, plan)
    spin_up(torch, launch)
    for _ in range(warmup):
        launch()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        launch()
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) * 1000.0 / steps


def time_cold(torch, ilpm, x, w, b, s, p, out, reps=20, scrub_mib=512):
    """Median µs of `reps` individually timed calls, each after a 512 MiB
    write that evicts the inputs, weights and output from L2 and the
    last-level cache (so every byte the call moves comes from or goes to
    HBM)."""
    launch = ilpm.conv2d_launcher(x, w, b, s, p, out)
    scrub = torch.empty(scrub_mib << 18, device="cuda", dtype=torch.float32)
    launch()
    times = []
    for i in range(reps):
        scrub.fill_(float(i))
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        launch()
        e.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(e) * 1000.0)
    del scrub
    times.sort()
    return times[len(times) // 2]


def time_winograd(torch, ilpm, x, w, b, p, out, steps, warmup):
    """Mean µs per call of the Winograd F(2x2,3x3) comparison path (filter
    transform done once beforehand), or None when it cannot run here."""
    try:
        u = ilpm.winograd_transform_filter(w)
        launch = ilpm.conv2d_winograd_launcher(x, u, b, p, out)
        for _ in range(warmup):
            launch()
    except ilpm.IlpmError:
        return None
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        launch()
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) * 1000.0 / steps


def cpu_baseline(case, x, w, b, y_gpu):
    """The CPU oracle timed on this host on the whole layer (repeated for at
    least 10 s),
    and the same run used as a parity spot check of the GPU output."""
    import numpy as np
    import oracle
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or min(16, os.cpu_count() or 1)
    used = oracle.set_threads(threads)
    flops, _, _, _ = layer_work(case.c_in, case.h, case.w, case.c_out, case.k, case.stride, case.pad,
                                b is not None)
    reps, elapsed = 0, 0.0
    ref = sab = None
    while elapsed < 10.0 and reps < 200:
        t0 = time.perf_counter()
        ref, sab = oracle.conv2d_f64(x, w, b, case.stride, case.pad)
        elapsed += time.perf_counter() - t0
        reps += 1
    ok, ratio, _ = oracle.check(y_gpu, ref, sab, case.c_in, case.k)
    # the same oracle on one thread, one run
    oracle.set_threads(1)
    t0 = time.perf_counter()
    oracle.conv2d_f64(x, w, b, case.stride, case.pad)
    one = time.perf_counter() - t0
    oracle.set_threads(used)
    return {"value": round(flops * reps / elapsed / 1e9, 3), "unit": "GFLOP/s", "cores": used,
            "kind": "oracle",
            "sample": f"whole layer, {reps} run(s), fp64 seven-loop oracle, {elapsed:.2f} s",
            "one_thread_gflops": round(flops / one / 1e9, 3),
            "host_cpu": _cpu_model(), "host_threads": os.cpu_count(),
            "parity_max_tol_ratio": round(ratio, 4), "parity_ok": bool(ok)}


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def measure_peaks(torch):
    """Measured ceilings: fp32 matrix-core and vector-FMA throughput (with the
    shader clock seen under the matrix-core load), HBM copy bandwidth, and the
    back-to-back cost of an empty launch."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "bench_peaks.so"))
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    res = {}

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / 1000.0 / reps

    iters = 4000
    for waves_per_simd in (1, 2):
        grid = 256 * waves_per_simd
        out = torch.empty(grid * 256, device="cuda")
        clk = torch.zeros(2 * grid, device="cuda", dtype=torch.int64)
        t = timed(lambda: lib.peak_mfma_launch(ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(clk.data_ptr()),
                                               iters, grid, st), 5)
        c = clk.view(-1, 2).double().cpu()
        mhz = float((c[:, 0] / (c[:, 1] / 100.0)).mean())
        res[f"mfma_f32_tflops_{waves_per_simd}w"] = round(grid * 4 * iters * 16 * 2048 / t / 1e12, 2)
        res[f"mfma_f32_clock_mhz_{waves_per_simd}w"] = round(mhz, 1)
    grid = 1024
    out = torch.empty(grid * 256, device="cuda")
    t = timed(lambda: lib.peak_valu_launch(ctypes.c_void_p(out.data_ptr()), iters, grid, st), 5)
    res["valu_fma_f32_tflops"] = round(grid * 256 * iters * 16 * 2 / t / 1e12, 2)
    n = 1 << 28  # 1 GiB of float32
    src = torch.ones(n, device="cuda")
    dst = torch.empty(n, device="cuda")
    t = timed(lambda: lib.copy_launch(ctypes.c_void_p(src.data_ptr()), ctypes.c_void_p(dst.data_ptr()),
                                      ctypes.c_size_t(n // 4), 4096, st), 10)
    res["hbm_copy_gbs"] = round(2 * 4 * n / t / 1e9, 1)
    del src, dst
    t = timed(lambda: lib.empty_launch(st), 2000)
    res["empty_launch_us"] = round(t * 1e6, 3)
    return res


def bench_case(torch, ilpm, case, steps, warmup, graph=False):
    from workloads import to_device
    x, w, b = case.inputs()
    xd, wd, bd = to_device(torch, x), to_device(torch, w), to_device(torch, b)
    plan = ilpm.plan(case.c_in, case.h, case.w, case.c_out, case.k, case.stride, case.pad)
    flops, nbytes, ho, wo = layer_work(case.c_in, case.h, case.w, case.c_out, case.k, case.stride, case.pad,
                                       b is not None)
    out = torch.empty((1, case.c_out, ho, wo), device="cuda", dtype=torch.float32)
    spin = {}
    us = time_layer(torch, ilpm, xd, wd, bd, case.stride, case.pad, out, steps, warmup, spin)
    res = dict(x=x, w=w, b=b, out=out, plan=plan, flops=flops, nbytes=nbytes, us=us, spin=spin)
    if graph:
        res["graph_us"] = time_layer_graph(torch, ilpm, xd, wd, bd, case.stride, case.pad, out, steps)
        res["prepacked_us"] = time_prepacked(torch, ilpm, xd, wd, bd, case.stride, case.pad, out, plan, steps,
                                             warmup)
        res["cold_us"] = time_cold(torch, ilpm, xd, wd, bd, case.stride, case.pad, out)
        if case.k == 3 and case.stride == 1:
            out_w = torch.empty_like(out)
            res["winograd_us"] = time_winograd(torch, ilpm, xd, wd, bd, case.pad, out_w, steps, warmup)
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=1000)
    ap.add_argument("--workload", default="vgg_early_64to64_224x224")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--spinup-ms", type=float, default=300.0,
                    help="untimed, wall-clock-bounded spin-up of each timed launch before its warm-up")
    ap.add_argument("--no-configs", action="store_true", help="only the headline layer (no per-config rows)")
    ap.add_argument("--all", action="store_true", help="also time every workload and the VGG-16 stack")
    ap.add_argument("--report", default=None, help="JSON file for the --all table")
    ap.add_argument("--peaks", action="store_true", help="also measure the MI355X ceilings")
    ap.add_argument("--copy-calib", type=int, default=0, metavar="MIB",
                    help="also run a plain copy of MIB MiB (counter calibration under rocprofv3)")
    ap.add_argument("--counter-run", action="store_true",
                    help="only the workload's spin-up, warm-up, timed and 20 cold calls (for rocprofv3 --pmc runs:"
                         " the dispatch counts are printed, so counter rows can be matched to the phases)")
    ap.add_argument("--lds-probe", action="store_true",
                    help="only run the LDS bank probe over lds_banks.probe_patterns() (for rocprofv3 --pmc)")
    ap.add_argument("--vgg16-stack", type=int, default=0, metavar="REPS",
                    help="only time the VGG-16 stack end to end, REPS passes per timing (kernel traces)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the library has no multi-GPU path "
              "(sharding of the batch-1 conv is a design note only)", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    import paper_1909_02765_amd as ilpm
    import workloads
    SPINUP["ms"] = max(0.0, args.spinup_ms)

    if args.lds_probe:
        print(json.dumps(run_lds_probe(torch)))
        return

    if args.vgg16_stack:
        rows = bench_vgg16_stack(torch, ilpm, workloads, args.vgg16_stack)
        print(json.dumps(rows))
        if any(r.get("same_output_bits") is False for r in rows):
            print("bench.py: a VGG-16 stack's output bits differ from its reference's", file=sys.stderr)
            sys.exit(1)
        return

    case = workloads.case_by_name(args.workload)
    if case is None:
        print(f"unknown workload {args.workload}", file=sys.stderr)
        sys.exit(2)

    if args.counter_run:
        r = bench_case(torch, ilpm, case, args.steps, args.warmup, graph=False)
        cold = time_cold(torch, ilpm, *(workloads.to_device(torch, t) for t in (r["x"], r["w"], r["b"])),
                         case.stride, case.pad, r["out"])
        print(json.dumps({"workload": case.name, "us_per_layer": round(r["us"], 3), "cold_us": round(cold, 3),
                          "dispatches": {"spinup": r["spin"]["calls"], "warmup": args.warmup, "timed": args.steps,
                                         "cold_first_uncounted": 1, "cold": 20},
                          "plan": ilpm.variant_name(r["plan"].path, r["plan"].variant) + f" x{r['plan'].splits}",
                          "kernel_digest": kernel_source_digest(),
                          "copy_calib_bytes_each_way": copy_calibration(torch, args.copy_calib) if args.copy_calib
                          else None}))
        return

    r = bench_case(torch, ilpm, case, args.steps, args.warmup, graph=True)
    us = r["us"]
    gflops = r["flops"] / (us * 1e-6) / 1e9
    floor_us, bound = roofline_floor_us(r["flops"], r["nbytes"])
    digest = kernel_source_digest()
    if bound == "mfma":
        roof = {"bound": "mfma", "achieved": round(r["flops"] / (us * 1e-6) / 1e12, 3),
                "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(r["nbytes"] / (us * 1e-6) / 1e9, 1),
                "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"] = measured_traffic(case.name, digest,
                                       ilpm.variant_name(r["plan"].path, r["plan"].variant) + f" x{r['plan'].splits}")
    roof["algorithmic_bytes"] = int(r["nbytes"])
    roof["floor_us"] = round(floor_us, 3)
    roof["kernel_digest"] = digest

    line = {
        "metric": METRIC, "value": round(gflops, 2), "unit": "GFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(us / 1000.0, 6),
        "us_per_layer": round(us, 3), "spinup_calls": r["spin"]["calls"], "spinup_ms": r["spin"]["ms"],
        "graph_replay_us_per_layer": round(r["graph_us"], 3),
        "prepacked_weights_us_per_layer": round(r["prepacked_us"], 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic (seeded SplitMix64 inputs, He-normal weights)",
        "config": {"workload": case.name, "input": [1, case.c_in, case.h, case.w],
                   "weights": [case.c_out, case.c_in, case.k, case.k], "stride": case.stride,
                   "pad": case.pad, "bias": r["b"] is not None, "parallelism": "none (1 GPU)",
                   "plan": r["plan"].as_dict()},
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        y = r["out"].cpu().numpy()
        line["cpu_baseline"] = cpu_baseline(case, r["x"], r["w"], r["b"], y)

    failures = []
    if not args.no_configs:
        line["configs"] = config_rows(torch, ilpm, workloads, case.name, failures)

    if args.copy_calib:
        line["copy_calib_bytes_each_way"] = copy_calibration(torch, args.copy_calib)

    if args.peaks:
        line["measured_peaks"] = measure_peaks(torch)
        print(json.dumps(line["measured_peaks"]), file=sys.stderr)

    if args.all:
        # Each row gets the default warm-up: after the host has spent a while
        # generating the next layer's inputs, the first few hundred calls
        # run ~8% slower (the GPU has idled).
        rows = []
        for c in workloads.ALL_CASES:
            rr = bench_case(torch, ilpm, c, max(200, args.steps // 4), 1000, graph=True)
            fl, kind = roofline_floor_us(rr["flops"], rr["nbytes"])
            rows.append({"layer": c.name, "us": round(rr["us"], 3), "graph_us": round(rr["graph_us"], 3),
                         "prepacked_us": round(rr["prepacked_us"], 3), "cold_us": round(rr["cold_us"], 3),
                         "cold_hbm_gbs": round(rr["nbytes"] / rr["cold_us"] / 1e3, 1),
                         "winograd_us": (round(rr["winograd_us"], 3) if rr.get("winograd_us") is not None
                                         else None),
                         "gflops": round(rr["flops"] / rr["us"] / 1e3, 1),
                         "floor_us": round(fl, 3), "bound": kind, "frac": round(fl / rr["us"], 4),
                         "plan": rr["plan"].as_dict()})
            rows[-1].update(prepacked_plan_row(torch, ilpm, c.c_in, c.h, c.w, c.c_out, c.k, c.stride, c.pad,
                                               rr["x"], rr["w"], rr["b"], rr["out"], max(200, args.steps // 4)))
            print(json.dumps(rows[-1]), file=sys.stderr)
        rows += bench_vgg16(torch, ilpm, workloads, max(200, args.steps // 10))
        if args.report:
            with open(args.report, "w") as f:
                json.dump(rows, f, indent=1)

    print(json.dumps(line), flush=True)
    if failures:
        print("bench.py: " + "; ".join(failures), file=sys.stderr)
        sys.exit(1)


CONFIG_ROWS = ["tiny_3to16_32x32", "resnet_conv4_256to256_14x14", "resnet_strided_128to256_28x28_s2",
               "deep_1x1_512to512_7x7", "deep_5x5_512to512_7x7"]


def copy_calibration(torch, mib):
    """Three plain copies of `mib` MiB (16-byte loads and stores): under
    rocprofv3 --pmc their FETCH_SIZE / WRITE_SIZE give the counters' scale
    for a known number of bytes.  Returns the bytes moved each way per copy."""
    import ctypes
    plib = ctypes.CDLL(os.path.join(ROOT, "bench_peaks.so"))
    n = mib << 18  # floats
    src = torch.ones(n, device="cuda")
    dst = torch.empty(n, device="cuda")
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    for _ in range(3):
        plib.copy_launch(ctypes.c_void_p(src.data_ptr()), ctypes.c_void_p(dst.data_ptr()),
                         ctypes.c_size_t(n // 4), 4096, st)
    torch.cuda.synchronize()
    return 4 * n


def config_rows(torch, ilpm, workloads, headline, failures, steps=500, warmup=200):
    """One compact row per other workload: µs per call (after the spin-up and
    warm-up), graph-replay µs, GFLOP/s, roofline bound / floor / fraction,
    and for HBM-bound rows the cold µs and its fraction; then the VGG-16 stack
    end to end and layer by layer."""
    rows = []
    for name in CONFIG_ROWS:
        if name == headline:
            continue
        c = workloads.case_by_name(name)
        x, w, b = c.inputs()
        xd, wd, bd = (workloads.to_device(torch, t) for t in (x, w, b))
        flops, nbytes, ho, wo = layer_work(c.c_in, c.h, c.w, c.c_out, c.k, c.stride, c.pad, b is not None)
        out = torch.empty((1, c.c_out, ho, wo), device="cuda", dtype=torch.float32)
        us = time_layer(torch, ilpm, xd, wd, bd, c.stride, c.pad, out, steps, warmup)
        gus = time_layer_graph(torch, ilpm, xd, wd, bd, c.stride, c.pad, out, steps)
        fl, kind = roofline_floor_us(flops, nbytes)
        plan = ilpm.plan(c.c_in, c.h, c.w, c.c_out, c.k, c.stride, c.pad)
        row = {"workload": name, "us": round(us, 3), "graph_us": round(gus, 3),
               "gflops": round(flops / us / 1e3, 1), "bound": kind, "floor_us": round(fl, 3),
               "frac": round(fl / us, 4), "plan": ilpm.variant_name(plan.path, plan.variant) + f" x{plan.splits}"}
        # The same layer on weights packed once beforehand for the plan
        # ilpm_conv2d_plan_prepacked picks (graph replay).
        pplan = ilpm.plan_prepacked(c.c_in, c.h, c.w, c.c_out, c.k, c.stride, c.pad)
        packed = ilpm.prepack_weights(wd, pplan)
        pus = time_graph(torch, lambda: ilpm.conv2d_prepacked_launcher(xd, packed, c.c_out, c.k, bd, c.stride, c.pad,
                                                                      out, pplan), steps)
        row["prepacked_graph_us"] = round(pus, 3)
        row["prepacked_plan"] = ilpm.variant_name(pplan.path, pplan.variant) + f" x{pplan.splits}"
        if kind == "hbm":
            cus = time_cold(torch, ilpm, xd, wd, bd, c.stride, c.pad, out)
            row["cold_us"] = round(cus, 3)
            row["cold_frac"] = round(fl / cus, 4)
        rows.append(row)
        print(json.dumps(row), file=sys.stderr)
    st = bench_vgg16_stack(torch, ilpm, workloads, 20)
    by = {r["layer"]: r for r in st}
    for r in st:
        if r.get("same_output_bits") is False:
            failures.append(f"{r['layer']}: output bits differ from its reference's")
    layers = bench_vgg16_layers(torch, ilpm, workloads, 200)
    floor_total = sum(l["floor_us"] for l in layers)
    flops_total = sum(l["gflop"] for l in layers) * 1e9
    us_f = by["vgg16_stack_fused"]["us"]
    rows.append({"workload": "vgg16_stack_13conv_224", "us": us_f,
                 "graph_us": by["vgg16_stack_fused_graph"]["us"], "unfused_us": by["vgg16_stack_unfused"]["us"],
                 "prepacked_us": by["vgg16_stack_fused_prepacked"]["us"],
                 "prepacked_graph_us": by["vgg16_stack_fused_prepacked_graph"]["us"],
                 "gflops": round(flops_total / us_f / 1e3, 1), "bound": "mfma (conv1_1 hbm)",
                 "floor_us": round(floor_total, 3), "frac": round(floor_total / us_f, 4),
                 "note": "end to end, fused ReLU / ReLU+2x2 max-pool epilogue, one call per conv",
                 "layers": [{k: l[k] for k in ("layer", "us", "frac")} for l in layers]})
    print(json.dumps(rows[-1]), file=sys.stderr)
    return rows


def bench_vgg16_layers(torch, ilpm, workloads, steps):
    """Each VGG-16 conv timed by itself (default plan, no epilogue) on the
    stack's own input to it."""
    from workloads import to_device
    out_rows = []
    x = to_device(torch, workloads.vgg16_input())
    for name, ci, co, hw, pool, seed in workloads.vgg16_layers():
        w = to_device(torch, workloads.vgg16_weights(ci, co, seed))
        out = torch.empty((1, co, hw, hw), device="cuda", dtype=torch.float32)
        us = time_layer(torch, ilpm, x, w, None, 1, 1, out, steps, 200)
        flops, nbytes, _, _ = layer_work(ci, hw, hw, co, 3, 1, 1, False)
        fl, kind = roofline_floor_us(flops, nbytes)
        out_rows.append({"layer": name, "us": round(us, 3), "frac": round(fl / us, 4), "floor_us": fl,
                         "gflop": flops / 1e9, "bound": kind})
        ilpm.relu_(out)
        x = ilpm.maxpool2x2(out) if pool else out
    return out_rows


def run_lds_probe(torch, iters=1000):
    """One lds_probe dispatch per address pattern of lds_banks.probe_patterns(),
    in order; returns the pattern names (the dispatch order, for matching the
    counter rows of a rocprofv3 run)."""
    import ctypes
    from paper_1909_02765_amd import lds_banks
    lib = ctypes.CDLL(os.path.join(ROOT, "bench_peaks.so"))
    out = torch.empty(64, device="cuda")
    names = []
    for name, width, table in lds_banks.probe_patterns():
        if len(table) != 64 or any(a < 0 or a + width > 16384 or a % width for a in table):
            raise ValueError(f"probe pattern {name} out of range")
        t = torch.tensor(table, dtype=torch.int32, device="cuda")
        rc = lib.lds_probe_launch(ctypes.c_void_p(t.data_ptr()), ctypes.c_void_p(out.data_ptr()), iters, width,
                                  ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        if rc != 0:
            raise RuntimeError(f"lds_probe_launch: {rc}")
        torch.cuda.synchronize()
        names.append(name)
    return {"lds_probe_iters": iters, "patterns": names}


def prepacked_plan_row(torch, ilpm, c_in, h, w_, c_out, k, s, p, x, w, b, out, steps):
    """The layer on weights packed once for ilpm_conv2d_plan_prepacked's plan:
    graph-replay µs and the plan's name."""
    from workloads import to_device
    x, w, b = (t if t is None or hasattr(t, "is_cuda") else to_device(torch, t) for t in (x, w, b))
    plan = ilpm.plan_prepacked(c_in, h, w_, c_out, k, s, p)
    packed = ilpm.prepack_weights(w, plan)
    us = time_graph(torch, lambda: ilpm.conv2d_prepacked_launcher(x, packed, c_out, k, b, s, p, out, plan), steps)
    return {"prepacked_plan_graph_us": round(us, 3),
            "prepacked_plan": ilpm.variant_name(plan.path, plan.variant) + f" x{plan.splits}"}


def bench_vgg16(torch, ilpm, workloads, steps):
    from workloads import to_device
    rows = []
    x = to_device(torch, workloads.vgg16_input())
    total_us = total_graph_us = total_floor = total_flops = 0.0
    for name, ci, co, hw, pool, seed in workloads.vgg16_layers():
        w = to_device(torch, workloads.vgg16_weights(ci, co, seed))
        out = torch.empty((1, co, hw, hw), device="cuda", dtype=torch.float32)
        us = time_layer(torch, ilpm, x, w, None, 1, 1, out, steps, 1000)
        gus = time_layer_graph(torch, ilpm, x, w, None, 1, 1, out, steps)
        flops, nbytes, _, _ = layer_work(ci, hw, hw, co, 3, 1, 1, False)
        fl, kind = roofline_floor_us(flops, nbytes)
        plan = ilpm.plan(ci, hw, hw, co, 3, 1, 1)
        rows.append({"layer": f"vgg16_{name}", "us": round(us, 3), "graph_us": round(gus, 3),
                     "gflops": round(flops / us / 1e3, 1),
                     "floor_us": round(fl, 3), "bound": kind, "frac": round(fl / us, 4), "plan": plan.as_dict()})
        rows[-1].update(prepacked_plan_row(torch, ilpm, ci, hw, hw, co, 3, 1, 1, x, w, None, out, steps))
        print(json.dumps(rows[-1]), file=sys.stderr)
        total_us += us
        total_graph_us += gus
        total_floor += fl
        total_flops += flops
        ilpm.relu_(out)
        x = ilpm.maxpool2x2(out) if pool else out
    rows += bench_vgg16_stack(torch, ilpm, workloads, max(20, steps // 10))
    rows.append({"layer": "vgg16_total_conv", "us": round(total_us, 3), "graph_us": round(total_graph_us, 3),
                 "gflops": round(total_flops / total_us / 1e3, 1), "floor_us": round(total_floor, 3),
                 "frac": round(total_floor / total_us, 4)})
    print(json.dumps(rows[-1]), file=sys.stderr)
    return rows


def bench_vgg16_stack(torch, ilpm, workloads, reps):
    """The whole 13-conv stack end to end (ReLU after every conv, 2x2 max-pool
    after stages 1-4), timed over `reps` back-to-back passes: once with the
    separate ReLU and pool kernels, once with the fused epilogue."""
    from workloads import to_device
    layers = workloads.vgg16_layers()
    x0 = to_device(torch, workloads.vgg16_input())
    ws = [to_device(torch, workloads.vgg16_weights(ci, co, seed)) for _, ci, co, _, _, seed in layers]
    # unfused: conv -> relu_ -> (pool)
    bufs, launches = [], []
    x = x0
    for (name, ci, co, hw, pool, _), w in zip(layers, ws):
        y = torch.empty((1, co, hw, hw), device="cuda", dtype=torch.float32)
        # the plan the fused call below picks for this layer's epilogue, so
        # that the two sequences round alike and must match bit for bit
        plan = ilpm.plan_for(ci, hw, hw, co, 3, 1, 1, ilpm.EPI_RELU | (ilpm.EPI_MAXPOOL2 if pool else 0))
        conv = ilpm.conv2d_launcher(x, w, None, 1, 1, y, plan=plan)
        launches.append(conv)
        launches.append(lambda y=y: ilpm.relu_(y))
        if pool:
            z = torch.empty((1, co, hw // 2, hw // 2), device="cuda", dtype=torch.float32)
            launches.append(lambda y=y, z=z: ilpm.lib.ilpm_maxpool2x2(
                ilpm._dev_f32(y, "y"), y.shape[1], y.shape[2], y.shape[3], ilpm._dev_f32(z, "z"),
                ilpm._stream_handle()))
            x = z
        else:
            x = y
        bufs.append(y)
    out_unfused = x
    # fused: one call per layer
    fused = []
    x = x0
    for (name, ci, co, hw, pool, _), w in zip(layers, ws):
        epi = ilpm.EPI_RELU | (ilpm.EPI_MAXPOOL2 if pool else 0)
        y = torch.empty(ilpm.epilogue_out_shape(co, hw, hw, 3, 1, 1, epi), device="cuda", dtype=torch.float32)
        fused.append(ilpm.conv2d_epilogue_launcher(x, w, None, 1, 1, epi, y))
        x = y
    out_fused = x

    def timed(fns):
        def one_pass():
            for f in fns:
                f()
        spin_up(torch, one_pass)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            for f in fns:
                f()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1000.0 / reps

    t_unfused = timed(launches)
    t_fused = timed(fused)
    same = bool(torch.equal(out_unfused, out_fused))
    ref = out_fused.clone()

    # The fused stack captured once in a HIP graph and replayed (no host
    # launch cost between layers); every replay's output is checked against
    # the eager result.  The eager passes above have sized the workspace, so
    # the library allocates nothing during capture.
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        fused_s = []
        x = x0
        for (name, ci, co, hw, pool, _), w in zip(layers, ws):
            epi = ilpm.EPI_RELU | (ilpm.EPI_MAXPOOL2 if pool else 0)
            y = torch.empty(ilpm.epilogue_out_shape(co, hw, hw, 3, 1, 1, epi), device="cuda", dtype=torch.float32)
            fused_s.append(ilpm.conv2d_epilogue_launcher(x, w, None, 1, 1, epi, y))
            x = y
        out_graph = x
        for f in fused_s:
            f()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for f in fused_s:
                f()
    torch.cuda.synchronize()
    spin_up(torch, g.replay)
    graph_same = True
    for _ in range(3):
        out_graph.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        graph_same = graph_same and bool(torch.equal(out_graph, ref))
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    t_graph = a.elapsed_time(b) * 1000.0 / reps
    out_graph.fill_(float("nan"))
    g.replay()
    torch.cuda.synchronize()
    graph_same = graph_same and bool(torch.equal(out_graph, ref))
    # The fused stack on prepacked weights: each layer on the plan
    # ilpm_conv2d_plan_for picks for its epilogue, its weights packed once beforehand
    # (outside the timed region, like loading a model).  Checked bit for bit
    # against the same plans run on the OIHW weights.
    pre, ref_pre = [], []
    x = xp = x0
    for (name, ci, co, hw, pool, _), w in zip(layers, ws):
        epi = ilpm.EPI_RELU | (ilpm.EPI_MAXPOOL2 if pool else 0)
        plan = ilpm.plan_for(ci, hw, hw, co, 3, 1, 1, epi, prepacked=True)
        packed = ilpm.prepack_weights(w, plan)
        y = torch.empty(ilpm.epilogue_out_shape(co, hw, hw, 3, 1, 1, epi), device="cuda", dtype=torch.float32)
        pre.append(ilpm.conv2d_prepacked_epilogue_launcher(xp, packed, co, 3, None, 1, 1, epi, y, plan))
        xr = ilpm.conv2d_epilogue(x, w, None, 1, 1, epi, plan=plan)
        ref_pre.append(xr)
        x, xp = xr, y
    out_pre = xp
    t_pre = timed(pre)
    pre_same = bool(torch.equal(out_pre, ref_pre[-1]))
    stream_p = torch.cuda.Stream()
    stream_p.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream_p):
        pre_s = []
        xp = x0
        for (name, ci, co, hw, pool, _), w in zip(layers, ws):
            epi = ilpm.EPI_RELU | (ilpm.EPI_MAXPOOL2 if pool else 0)
            plan = ilpm.plan_for(ci, hw, hw, co, 3, 1, 1, epi, prepacked=True)
            packed = ilpm.prepack_weights(w, plan)
            y = torch.empty(ilpm.epilogue_out_shape(co, hw, hw, 3, 1, 1, epi), device="cuda", dtype=torch.float32)
            pre_s.append(ilpm.conv2d_prepacked_epilogue_launcher(xp, packed, co, 3, None, 1, 1, epi, y, plan))
            xp = y
        out_pre_graph = xp
        for f in pre_s:
            f()
        torch.cuda.synchronize()
        gp = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gp, stream=stream_p):
            for f in pre_s:
                f()
    torch.cuda.synchronize()
    spin_up(torch, gp.replay)
    for _ in range(3):
        out_pre_graph.fill_(float("nan"))
        gp.replay()
        torch.cuda.synchronize()
        pre_same = pre_same and bool(torch.equal(out_pre_graph, out_pre))
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        gp.replay()
    b.record()
    torch.cuda.synchronize()
    t_pre_graph = a.elapsed_time(b) * 1000.0 / reps
    rows = [{"layer": "vgg16_stack_unfused", "us": round(t_unfused, 3),
             "note": "13 convs + 13 ReLU + 4 max-pool kernels, end to end"},
            {"layer": "vgg16_stack_fused", "us": round(t_fused, 3),
             "note": "13 convs with the fused ReLU / ReLU+max-pool epilogue", "same_output_bits": same},
            {"layer": "vgg16_stack_fused_graph", "us": round(t_graph, 3),
             "note": "the fused stack replayed from one captured HIP graph", "same_output_bits": graph_same},
            {"layer": "vgg16_stack_fused_prepacked", "us": round(t_pre, 3),
             "note": "the fused stack on weights prepacked once for ilpm_conv2d_plan_for's plans "
                     "(bits equal the same plans on OIHW weights)", "same_output_bits": pre_same},
            {"layer": "vgg16_stack_fused_prepacked_graph", "us": round(t_pre_graph, 3),
             "note": "the prepacked fused stack replayed from one captured HIP graph",
             "same_output_bits": pre_same}]
    for r in rows:
        print(json.dumps(r), file=sys.stderr)
    return rows


if __name__ == "__main__":
    main()
