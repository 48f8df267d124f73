"""Benchmark of the conv2d forward primitive on one MI355X.

Default workload: fp32 NCHW conv2d, N=32, C=K=64, 56x56, 3x3, stride 1, pad 1
(the contraction-bound square-channel layer), AUTO algorithm (implicit GEMM).
A step is one conv2d_fwd over the whole batch with inputs resident in HBM.

Prints ONE JSON line with the throughput (TFLOP/s), the dominant kernel's
roofline position (its duration from the HIP events that enclose every phase
launch in the timed region), the per-phase breakdown of the timed region, the
explicit im2col path's pack-phase time share on the same workload, and the
CPU oracle timed on a bounded sample of the same workload.

    python bench.py [--gpus 1] [--steps 50] [--warmup 10] [--workload cfg2] [--no-cpu]
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "conv2d TFLOP/s and % of MFMA/HBM roofline per shape; pack-phase time share"
PEAK_TFLOPS = {"f32": 157.3, "bf16": 2516.6}   # dense MFMA
PEAK_HBM_GBS = 8000.0
# fp32 FMA on the vector ALU without packed instructions (the build disables them):
# 256 CUs x 4 SIMDs x 16 lanes x 2 flops x 2.4 GHz
PEAK_VALU_TFLOPS = 78.6
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
# the kernels' sources and the planner's (which picks the instantiation, tile and launch shape)
_PLANNER = ["paper_2407_10730_amd/csrc/conv2d_api.hip", "paper_2407_10730_amd/csrc/conv2d_internal.h"]
KERNEL_SOURCES = {
    "implicit_gemm": ["paper_2407_10730_amd/csrc/gemm_mfma.hip", "paper_2407_10730_amd/csrc/pack_kernels.hip",
                      "paper_2407_10730_amd/csrc/slice_conv.hip"] + _PLANNER,
    "im2col_gemm": ["paper_2407_10730_amd/csrc/gemm_mfma.hip", "paper_2407_10730_amd/csrc/pack_kernels.hip"] + _PLANNER,
    "direct": ["paper_2407_10730_amd/csrc/direct_kernels.hip"] + _PLANNER,
}


def kernel_hash(algo_name):
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[algo_name]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def describe(cs):
    return (f"conv2d fwd {cs.layout.upper()} {cs.x_dtype}->{cs.y_dtype} N{cs.n} C{cs.c} {cs.h}x{cs.w} "
            f"K{cs.k} {cs.r}x{cs.s} s{cs.stride[0]}x{cs.stride[1]} p{cs.pad[0]}x{cs.pad[1]} "
            f"d{cs.dil[0]}x{cs.dil[1]} g{cs.groups}{' +bias' if cs.has_bias else ''}")


def algorithmic_bytes(cs, nkhw):
    """Bytes the operation must move at least once: the input pixels its windows touch,
    the weights, the bias and the output."""
    n, k, ho, wo = nkhw
    xs = 2 if cs.x_dtype == "bf16" else 4
    ys = 2 if cs.y_dtype == "bf16" else 4
    rows = set()
    for o in range(ho):
        for r in range(cs.r):
            h = o * cs.stride[0] - cs.pad[0] + r * cs.dil[0]
            if 0 <= h < cs.h:
                rows.add(h)
    cols = set()
    for o in range(wo):
        for s in range(cs.s):
            w = o * cs.stride[1] - cs.pad[1] + s * cs.dil[1]
            if 0 <= w < cs.w:
                cols.add(w)
    x_touched = n * cs.c * len(rows) * len(cols) * xs
    w_bytes = k * (cs.c // cs.groups) * cs.r * cs.s * xs
    b_bytes = 4 * k if cs.has_bias else 0
    return x_touched + w_bytes + b_bytes + n * k * ho * wo * ys


def load_traffic(workload, algo_name):
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    ent = data.get(f"{workload}:{algo_name}")
    if not ent or ent.get("kernel_hash") != kernel_hash(algo_name):
        return None
    return ent.get("bytes_per_launch")


def cpu_baseline(cs, x, w, b, y_gpu, flops_per_image, target_s=10.0):
    """Time the fp64 oracle on the first images of the batch (host cores) and
    compare the GPU output on them."""
    import numpy as np
    import oracle
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or len(os.sched_getaffinity(0))
    threads = max(1, min(threads, len(os.sched_getaffinity(0))))
    bias = b if cs.has_bias else None
    t0 = time.perf_counter()
    oracle.conv2d(x[:1], w, bias, cs.stride, cs.pad, cs.dil, cs.groups, nthreads=threads, want_abs=False)
    t1 = time.perf_counter() - t0
    n_img = int(max(1, min(cs.n, round(target_s / max(t1, 1e-6)))))
    t0 = time.perf_counter()
    y_ref, a_ref = oracle.conv2d(x[:n_img], w, bias, cs.stride, cs.pad, cs.dil, cs.groups, nthreads=threads)
    dt = time.perf_counter() - t0
    lit, pt = oracle.normalised_errors(y_gpu[:n_img], y_ref, a_ref)
    # a whole batch that takes well under the target is timed over repeated passes
    passes = 1
    if n_img == cs.n and dt < 0.5 * target_s:
        passes = int(min(100, max(2, round(target_s / max(dt, 1e-6)))))
        t0 = time.perf_counter()
        for _ in range(passes):
            oracle.conv2d(x[:n_img], w, bias, cs.stride, cs.pad, cs.dil, cs.groups, nthreads=threads,
                          want_abs=False)
        dt = (time.perf_counter() - t0) / passes
    # one image on one thread as well, as the paper's single-thread protocol times the CPU
    t0 = time.perf_counter()
    oracle.conv2d(x[:1], w, bias, cs.stride, cs.pad, cs.dil, cs.groups, nthreads=1, want_abs=False)
    dt1 = time.perf_counter() - t0
    res = {
        "value": flops_per_image * n_img / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"fp64 seven-loop oracle over the first {n_img} of {cs.n} images (all outputs)"
                  + (f", {passes} passes" if passes > 1 else "") + f", {dt * passes:.2f} s wall",
        "seconds": dt * passes,
        "passes": passes,
        "cpu_model": _cpu_model(),
        "single_thread": {"value": flops_per_image / dt1 / 1e12, "unit": "TFLOP/s", "cores": 1,
                          "sample": "first image", "seconds": dt1},
    }
    return res, {"images": n_img, "err_per_point": pt, "err_literal": lit}


def cpu_im2col_gemm(cs, x, w, b, flops_per_image, n_img=1):
    """Context beside the oracle: the paper's baseline algorithm (explicit im2col, then one
    GEMM) on the host in fp32 with numpy's BLAS, timed on the first images."""
    import numpy as np
    from numpy.lib.stride_tricks import sliding_window_view
    n_img = max(1, min(n_img, cs.n))
    g = cs.groups
    sh, sw = cs.stride
    ph, pw = cs.pad
    dh, dw = cs.dil
    xs = np.ascontiguousarray(x[:n_img], dtype=np.float32)
    wf = np.ascontiguousarray(w, dtype=np.float32)
    t0 = time.perf_counter()
    xp = np.pad(xs, ((0, 0), (0, 0), (ph, ph), (pw, pw)))
    eh, ew = (cs.r - 1) * dh + 1, (cs.s - 1) * dw + 1
    win = sliding_window_view(xp, (eh, ew), axis=(2, 3))[:, :, ::sh, ::sw, ::dh, ::dw]  # N C Ho Wo R S
    n, c, ho, wo, r, s_ = win.shape
    cg, kg = c // g, cs.k // g
    ys = []
    for gi in range(g):
        col = win[:, gi * cg:(gi + 1) * cg].transpose(1, 4, 5, 0, 2, 3).reshape(cg * r * s_, n * ho * wo)
        ys.append(wf[gi * kg:(gi + 1) * kg].reshape(kg, cg * r * s_) @ col)
    y = np.concatenate(ys, axis=0).reshape(cs.k, n, ho, wo).transpose(1, 0, 2, 3)
    if cs.has_bias:
        y = y + b.astype(np.float32)[None, :, None, None]
    dt = time.perf_counter() - t0
    return {"value": flops_per_image * n_img / dt / 1e12, "unit": "TFLOP/s", "kind": "numpy im2col + BLAS GEMM, fp32",
            "sample": f"first {n_img} of {cs.n} images", "seconds": dt}, y


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def time_algo(dc, algo, steps, warmup, B, torch, timing):
    """Warm up, then time exactly `steps` calls bracketed by device synchronisation, with an
    event pair on the launch stream around the timed calls.  timing = CONV2D_TIMING_OFF for
    the timed loops (no events between kernels), or CONV2D_TIMING_PHASES for the breakdown
    loop (an event pair around every phase launch).  Returns (wall seconds, event ms per
    step, breakdown or None)."""
    stream = torch.cuda.current_stream()
    B.conv2d_set_timing(dc.desc, timing)
    for _ in range(warmup):
        dc.run(algo, stream)
    torch.cuda.synchronize()
    B.conv2d_breakdown_reset(dc.desc)
    torch.cuda.synchronize()
    ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ea.record(stream)
    for _ in range(steps):
        dc.run(algo, stream)
    eb.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    bd = dc.breakdown(algo) if timing == B.CONV2D_TIMING_PHASES else None
    B.conv2d_set_timing(dc.desc, B.CONV2D_TIMING_OFF)
    return wall, ea.elapsed_time(eb) / steps, bd


def clock_ramp(dc, algo, seconds, torch):
    """Run the workload back to back for a fixed time before anything is counted: the GPU's
    clocks take a few milliseconds of load to come up, more than a handful of warm-up calls."""
    stream = torch.cuda.current_stream()
    calls = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(10):
            dc.run(algo, stream)
        calls += 10
        torch.cuda.synchronize()
    return {"seconds": time.perf_counter() - t0, "calls": calls}


def launches_per_step(dc, algo, B, torch):
    """Kernel launches of one call (every phase launch once), from one PHASES-mode call."""
    B.conv2d_set_timing(dc.desc, B.CONV2D_TIMING_PHASES)
    B.conv2d_breakdown_reset(dc.desc)
    dc.run(algo)
    torch.cuda.synchronize()
    bd = dc.breakdown(algo)
    B.conv2d_set_timing(dc.desc, B.CONV2D_TIMING_OFF)
    B.conv2d_breakdown_reset(dc.desc)
    return sum(v for p, v in bd["calls"].items() if p != "pre_analysis"), bd


def kernel_duration(dc, algo, event_ms_per_step, B, torch):
    """Average duration of the step's dominant kernel from an event pair on its stream around
    back-to-back launches of that kernel alone: the timed loop's own events when a step is that
    one launch, else the kernel probe (the implicit microkernel without the launches around
    it).  Returns (ms, source) or (None, reason)."""
    launches, bd = launches_per_step(dc, algo, B, torch)
    if launches == 1:
        return event_ms_per_step, "timed loop (one launch per step)"
    if algo == B.CONV2D_ALGO_IMPLICIT_GEMM and bd["calls"]["in_microkernel"] == 1:
        stream = torch.cuda.current_stream()
        ms = time_launches(lambda: B.conv2d_kernel_probe(dc.desc, dc.x, dc.w, dc.b, dc.y, stream), 50, torch)
        # restore y: the probe may leave split partials only
        dc.run(algo, stream)
        torch.cuda.synchronize()
        return ms, "kernel probe (microkernel alone, back to back)"
    return None, f"{launches} launches per step and no single-kernel probe for this algorithm"


def cold_median(dc, algo, runs, B, torch):
    """Median of single calls with the 256 MB last-level cache flushed before each (the
    library's copy probe moves 512 MiB through it, outside the timed events)."""
    stream = torch.cuda.current_stream()
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    B.conv2d_set_timing(dc.desc, B.CONV2D_TIMING_TOTAL)
    B.conv2d_breakdown_reset(dc.desc)
    times = []
    for _ in range(runs):
        B.conv2d_probe_copy(flush[256 << 20:], flush[:256 << 20], 256 << 20, stream)
        torch.cuda.synchronize()
        before = dc.breakdown(algo)["total_ms"] if times else 0.0
        dc.run(algo, stream)
        torch.cuda.synchronize()
        after = dc.breakdown(algo)["total_ms"]
        times.append(after - before)
    del flush
    B.conv2d_set_timing(dc.desc, B.CONV2D_TIMING_OFF)
    times.sort()
    return times[len(times) // 2]


def time_launches(launch, reps, torch):
    """Average duration of `launch()` (one kernel on the current stream) over `reps`
    back-to-back launches, from an event pair on that stream."""
    stream = torch.cuda.current_stream()
    for _ in range(3):
        launch()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(reps):
        launch()
    b.record(stream)
    b.synchronize()
    return a.elapsed_time(b) / reps


def kernel_label(plan, B):
    """Microkernel name, with its tile where it has one (the direct kernels have none)."""
    name = B.KERNEL_NAMES[plan.kernel]
    return f"{name} {plan.tile_m}x{plan.tile_n}" if plan.tile_m > 0 else name


def roofline(cs, nkhw, flops, kern_ms):
    """Which roofline bounds the operation (MFMA when the arithmetic intensity on algorithmic
    bytes reaches the dtype's ridge point; the vector ALU for direct grouped kernels whose
    intensity outruns it; HBM otherwise) and the kernel's fraction of it."""
    xdt = cs.x_dtype
    alg_bytes = algorithmic_bytes(cs, nkhw)
    ai = flops / alg_bytes
    ridge = PEAK_TFLOPS[xdt] * 1e12 / (PEAK_HBM_GBS * 1e9)
    out = {"algorithmic_bytes": alg_bytes, "algorithmic_flops": flops, "arith_intensity": ai}
    if kern_ms is None:
        out.update({"bound": None, "achieved": None, "peak": None, "unit": None, "frac": None})
        return out
    if ai >= ridge:
        achieved = flops / (kern_ms * 1e-3) / 1e12
        out.update({"bound": "mfma", "achieved": achieved, "peak": PEAK_TFLOPS[xdt], "unit": "TFLOP/s",
                    "frac": achieved / PEAK_TFLOPS[xdt]})
    elif cs.groups > 1 and ai * PEAK_HBM_GBS * 1e9 > PEAK_VALU_TFLOPS * 1e12:
        achieved = flops / (kern_ms * 1e-3) / 1e12
        out.update({"bound": "alu", "achieved": achieved, "peak": PEAK_VALU_TFLOPS, "unit": "TFLOP/s",
                    "frac": achieved / PEAK_VALU_TFLOPS})
    else:
        achieved = alg_bytes / (kern_ms * 1e-3) / 1e9
        out.update({"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": achieved / PEAK_HBM_GBS})
    return out


def measured_peaks(B, torch):
    """The roofline probes: MFMA issue rate (fp32, bf16) on register operands and the
    device copy rate (read + write bytes), next to the published peaks."""
    stream = torch.cuda.current_stream()
    sink = torch.empty(1 << 20, dtype=torch.float32, device="cuda")
    out = {}
    for name, dt, iters in (("mfma_f32_tflops", B.CONV2D_F32, 20000), ("mfma_bf16_tflops", B.CONV2D_BF16, 40000)):
        flops = [0.0]

        def run(dt=dt, iters=iters):
            flops[0] = B.conv2d_probe_mfma(dt, iters, sink, stream)
        ms = time_launches(run, 5, torch)
        out[name] = flops[0] / (ms * 1e-3) / 1e12
    buf = torch.empty(2 << 30, dtype=torch.uint8, device="cuda")
    src, dst = buf[: 1 << 30], buf[1 << 30:]
    ms = time_launches(lambda: B.conv2d_probe_copy(dst, src, 1 << 30, stream), 5, torch)
    out["copy_gbs"] = 2 * (1 << 30) / (ms * 1e-3) / 1e9
    del buf, sink
    out["published"] = {"mfma_f32_tflops": PEAK_TFLOPS["f32"], "mfma_bf16_tflops": PEAK_TFLOPS["bf16"],
                        "hbm_gbs": PEAK_HBM_GBS}
    return out


PROFILE_COMMANDS = {
    "trace": "rocprofv3 --kernel-trace --stats -f csv -d {d}/trace -o run -- python -u bench.py --no-cpu --no-pack-probe "
             "--no-per-config --workload {w}",
    "pmc1": "rocprofv3 --pmc SQ_WAVES SQ_BUSY_CYCLES SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU SQ_INSTS_MFMA "
            "SQ_LDS_BANK_CONFLICT GRBM_GUI_ACTIVE -f csv -d {d}/pmc1 -o run -- python -u bench.py --no-cpu --no-pack-probe "
            "--no-per-config --ramp-seconds 0.2 --steps 5 --warmup 1 --cold-runs 1 --workload {w}",
    "pmc2": "rocprofv3 --pmc FETCH_SIZE -f csv -d {d}/pmc2 -o run -- python -u bench.py --no-cpu --no-pack-probe "
            "--no-per-config --ramp-seconds 0.2 --steps 5 --warmup 1 --cold-runs 1 --calibrate-copy --workload {w}",
    "pmc3": "rocprofv3 --pmc WRITE_SIZE -f csv -d {d}/pmc3 -o run -- python -u bench.py --no-cpu --no-pack-probe "
            "--no-per-config --ramp-seconds 0.2 --steps 5 --warmup 1 --cold-runs 1 --calibrate-copy --workload {w}",
}


def summarize_profiles(d, workload, algo_name="implicit_gemm"):
    """Turn the rocprofv3 CSV outputs of PROFILE_COMMANDS into the short text summaries
    kept under profiles/ and the per-launch HBM traffic in profiles/traffic.json."""
    import csv
    import collections

    def rows(path):
        with open(path) as f:
            return list(csv.DictReader(f))

    def short(name):
        return name.split("(")[0].replace("void ", "")[:90]

    lines = [f"# rocprofv3 summary: workload {workload}", ""]
    stats = rows(os.path.join(d, "trace", "run_kernel_stats.csv"))
    lines += ["## kernel trace (--kernel-trace --stats)", "",
              "command (from the repository root on the GPU box): `"
              + PROFILE_COMMANDS["trace"].format(d="gpurun_out/<dir>", w=workload) + "`", "",
              "| kernel | calls | avg us | min us | max us | share % |", "|---|---|---|---|---|---|"]
    for r in stats:
        lines.append(f"| `{short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs'])/1e3:.1f} | "
                     f"{float(r['MinNs'])/1e3:.1f} | {float(r['MaxNs'])/1e3:.1f} | {float(r['Percentage']):.1f} |")
    counters = collections.defaultdict(lambda: collections.defaultdict(list))
    for sub in ("pmc1", "pmc2", "pmc3"):
        path = os.path.join(d, sub, "run_counter_collection.csv")
        if not os.path.exists(path):
            continue
        for r in rows(path):
            counters[(r["Kernel_Name"], r["Grid_Size"])][r["Counter_Name"]].append(float(r["Counter_Value"]))
    # calibration: the 1 GiB device copy
    cal_f = cal_w = None
    # (only the dispatches of that size: the same kernel also runs small copies)
    for (name, grid), cs in counters.items():
        if "copyBuffer" not in name:
            continue
        big_f = [v for v in cs.get("FETCH_SIZE", []) if v > 400000]
        big_w = [v for v in cs.get("WRITE_SIZE", []) if v > 400000]
        if big_f:
            cal_f = (1 << 20) / (sum(big_f) / len(big_f))
        if big_w:
            cal_w = (1 << 20) / (sum(big_w) / len(big_w))
    lines += ["", "## counters per kernel (mean per dispatch)", ""]
    for k in ("pmc1", "pmc2", "pmc3"):
        lines.append("command: `" + PROFILE_COMMANDS[k].format(d="gpurun_out/<dir>", w=workload) + "`")
    lines += ["", f"HBM byte scale factors from the 1 GiB device copy: FETCH_SIZE x {cal_f}, WRITE_SIZE x {cal_w}"
              " (counters are in KiB per dispatch)", ""]
    traffic = {}
    for (name, grid), cs in sorted(counters.items()):
        if "cv::" not in name:
            continue
        mean = {c: sum(v) / len(v) for c, v in cs.items()}
        txt = ", ".join(f"{c}={v:.0f}" for c, v in sorted(mean.items()))
        lines.append(f"- `{short(name)}` grid {grid}: {txt}")
        if "FETCH_SIZE" in mean and "WRITE_SIZE" in mean and cal_f and cal_w:
            b = mean["FETCH_SIZE"] * 1024 * cal_f + mean["WRITE_SIZE"] * 1024 * cal_w
            traffic[short(name)] = b
            lines.append(f"  - HBM traffic per dispatch: {b/1e6:.2f} MB (fetch {mean['FETCH_SIZE']*1024*cal_f/1e6:.2f}"
                         f" + write {mean['WRITE_SIZE']*1024*cal_w/1e6:.2f})")
        if "SQ_VALU_MFMA_BUSY_CYCLES" in mean and "GRBM_GUI_ACTIVE" in mean:
            busy = mean["SQ_VALU_MFMA_BUSY_CYCLES"] / 1024 / (mean["GRBM_GUI_ACTIVE"] / 8)
            lines.append(f"  - MFMA busy fraction (busy cycles per SIMD / active cycles per XCD): {busy:.3f}")
    return "\n".join(lines) + "\n", traffic


def run_sweep(report_path, B, torch):
    """Time every convolution of the 500-convolution sweep with the planner's algorithm and
    report, per class, the fraction of the MFMA roofline (contraction-bound: arithmetic
    intensity at or above the ridge) or of the HBM roofline (the rest)."""
    import datagen
    from paper_2407_10730_amd.runner import DeviceConv, params_for

    def out_hw(cs):
        d = B.conv2d_desc_create(params_for(cs))
        try:
            return B.conv2d_output_shape(d)[2:]
        finally:
            B.conv2d_desc_destroy(d)

    shapes, rejected = datagen.sweep_shapes(out_hw)
    dev = torch.device("cuda:0")
    rows = []
    for cs in shapes:
        x = datagen.draw_torch(cs.seed, datagen.TENSOR_X, cs.x_shape(), device=dev)
        w = datagen.draw_torch(cs.seed, datagen.TENSOR_W, cs.w_shape(), device=dev)
        b = datagen.draw_torch(cs.seed, datagen.TENSOR_B, (cs.k,), device=dev)
        if cs.x_dtype == "bf16":
            x, w = x.to(torch.bfloat16), w.to(torch.bfloat16)
        dc = DeviceConv(cs, device_inputs=(x, w, b))
        B.conv2d_set_timing(dc.desc, B.CONV2D_TIMING_OFF)
        stream = torch.cuda.current_stream()
        dc.run(B.CONV2D_ALGO_AUTO, stream)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        dc.run(B.CONV2D_ALGO_AUTO, stream)
        torch.cuda.synchronize()
        t1 = time.perf_counter() - t0
        runs = int(min(20, max(3, 0.05 / max(t1, 1e-6))))
        t0 = time.perf_counter()
        for _ in range(runs):
            dc.run(B.CONV2D_ALGO_AUTO, stream)
        torch.cuda.synchronize()
        sec = (time.perf_counter() - t0) / runs
        n, k, ho, wo = dc.out_nkhw
        flops = 2 * n * k * (cs.c // cs.groups) * cs.r * cs.s * ho * wo
        nbytes = algorithmic_bytes(cs, dc.out_nkhw)
        ai = flops / nbytes
        peak = PEAK_TFLOPS[cs.x_dtype]
        ridge = peak * 1e12 / (PEAK_HBM_GBS * 1e9)
        tf = flops / sec / 1e12
        gbs = nbytes / sec / 1e9
        if ai >= ridge:
            bound, frac, t_roof = "mfma", tf / peak, flops / (peak * 1e12)
        elif cs.groups > 1 and ai * PEAK_HBM_GBS * 1e9 > PEAK_VALU_TFLOPS * 1e12:
            # the direct kernel computes on the vector ALU: large filters in bf16 outrun it
            bound, frac, t_roof = "alu", tf / PEAK_VALU_TFLOPS, flops / (PEAK_VALU_TFLOPS * 1e12)
        else:
            bound, frac, t_roof = "hbm", gbs / PEAK_HBM_GBS, nbytes / (PEAK_HBM_GBS * 1e9)
        algo = B.ALGO_NAMES[dc.plan(B.CONV2D_ALGO_AUTO).algo]
        rows.append({"name": cs.name, "dtype": cs.x_dtype, "n": cs.n, "c": cs.c, "hw": cs.h, "k": cs.k,
                     "r": cs.r, "stride": cs.stride[0], "dil": cs.dil[0], "groups": cs.groups,
                     "algo": algo, "us": sec * 1e6, "tflops": tf, "gbs": gbs, "ai": ai, "bound": bound,
                     "frac": frac, "roofline_us": t_roof * 1e6, "depthwise": cs.groups > 1})
        dc.close()
        del x, w, b
    def summary(sel):
        if not sel:
            return None
        fr = sorted(r["frac"] for r in sel)
        return {"count": len(sel), "median_frac": fr[len(fr) // 2], "min_frac": fr[0], "max_frac": fr[-1]}
    # a convolution whose roofline time is a few microseconds is bound by the launch and the
    # kernel's fixed start-up; the "large" summaries keep those with >= 20 us of roofline time
    big = [r for r in rows if r["roofline_us"] >= 20.0]
    out = {
        "rejected_draws": rejected,
        "contraction_bound_f32": summary([r for r in rows if r["bound"] == "mfma" and r["dtype"] == "f32"]),
        "contraction_bound_bf16": summary([r for r in rows if r["bound"] == "mfma" and r["dtype"] == "bf16"]),
        "depthwise": summary([r for r in rows if r["depthwise"]]),
        "depthwise_alu_bound": summary([r for r in rows if r["depthwise"] and r["bound"] == "alu"]),
        "hbm_bound_other": summary([r for r in rows if r["bound"] == "hbm" and not r["depthwise"]]),
        "large_contraction_bound_f32": summary([r for r in big if r["bound"] == "mfma" and r["dtype"] == "f32"]),
        "large_contraction_bound_bf16": summary([r for r in big if r["bound"] == "mfma" and r["dtype"] == "bf16"]),
        "large_depthwise": summary([r for r in big if r["depthwise"]]),
        "large_hbm_bound_other": summary([r for r in big if r["bound"] == "hbm" and not r["depthwise"]]),
        "depthwise_at_70pct_hbm": sum(1 for r in rows if r["depthwise"] and r["bound"] == "hbm" and r["frac"] >= 0.7),
        "contraction_at_60pct_mfma": sum(1 for r in rows if r["bound"] == "mfma" and r["frac"] >= 0.6),
        "total_seconds_one_pass": sum(r["us"] for r in rows) * 1e-6,
    }
    with open(report_path, "w") as f:
        json.dump({"summary": out, "convs": rows}, f, indent=1)
    return out


PER_CONFIG = ["cfg1", "cfg2", "cfg3a", "cfg3b", "cfg4", "cfg4_bf16", "dw", "dw_bf16", "grp_g64", "grp_g32",
              "bf16_3x3"]
# the oracle evaluated on every output (the other rows: sampled outputs), and single-threaded
ORACLE_FULL = {"cfg1", "cfg2", "cfg3a", "cfg3b", "cfg4", "cfg4_bf16"}
ORACLE_SINGLE_THREAD = {"cfg1", "cfg2"}


def config_gpu(name, args, B, torch):
    """GPU half of one per-shape row: step time, kernel time, roofline position, the explicit
    path's pack share; the output is kept on the host for the oracle half."""
    import datagen
    from paper_2407_10730_amd.runner import DeviceConv
    cs = datagen.CONFIGS[name]
    print(f"[bench] per-config {name}: {describe(cs)}", file=sys.stderr, flush=True)
    dc = DeviceConv(cs)
    try:
        n, k, ho, wo = dc.out_nkhw
        flops = 2 * n * k * (cs.c // cs.groups) * cs.r * cs.s * ho * wo
        algo = dc.plan(B.CONV2D_ALGO_AUTO).algo
        plan = dc.plan(algo)
        clock_ramp(dc, algo, 0.15, torch)
        wall, _, _ = time_algo(dc, algo, 3, 0, B, torch, B.CONV2D_TIMING_OFF)
        steps = int(max(args.steps, min(2000, 0.03 / max(wall / 3, 1e-7))))
        wall, ev_ms, _ = time_algo(dc, algo, steps, args.warmup, B, torch, B.CONV2D_TIMING_OFF)
        ms = wall * 1e3 / steps
        kern_ms, src = kernel_duration(dc, algo, ev_ms, B, torch)
        roof = roofline(cs, dc.out_nkhw, flops, kern_ms)
        roof["kernel_us"] = None if kern_ms is None else kern_ms * 1e3
        roof["kernel_source"] = src
        roof["traffic"] = load_traffic(name, B.ALGO_NAMES[algo])
        _, _, bd = time_algo(dc, algo, 5, 1, B, torch, B.CONV2D_TIMING_PHASES)
        row = {"workload": describe(cs), "algo": B.ALGO_NAMES[algo],
               "kernel": kernel_label(plan, B),
               "steps": steps, "ms_per_step": ms, "event_ms_per_step": ev_ms,
               "tflops": flops / (ms * 1e-3) / 1e12, "roofline": roof,
               "kernel_le_step": None if kern_ms is None else kern_ms <= max(ms, ev_ms) * 1.02,
               "breakdown_ms_per_call": {p: v / 5 for p, v in bd["ms"].items() if p != "pre_analysis"}}
        # the explicit im2col path on the same operation: its packing share of the time
        try:
            dc.plan(B.CONV2D_ALGO_IM2COL_GEMM)
            ok = True
        except B.Conv2dError:
            ok = False
        if ok:
            wall_e, _, _ = time_algo(dc, B.CONV2D_ALGO_IM2COL_GEMM, 5, 2, B, torch, B.CONV2D_TIMING_OFF)
            _, _, bd_e = time_algo(dc, B.CONV2D_ALGO_IM2COL_GEMM, 5, 1, B, torch, B.CONV2D_TIMING_PHASES)
            opsum = sum(v for p, v in bd_e["ms"].items() if p != "pre_analysis")
            row["explicit_im2col"] = {"ms_per_step": wall_e * 1e3 / 5,
                                      "pack_share": bd_e["ms"]["in_packing"] / opsum if opsum > 0 else None,
                                      "t_explicit_over_t_main": wall_e * 1e3 / 5 / ms}
            dc.run(algo)   # y back to the main algorithm's result
            torch.cuda.synchronize()
        y = dc.y_nchw()
        host = (dc.x_host, dc.w_host, dc.b_host)
    finally:
        dc.close()
    return row, (cs, y, host, flops)


def config_oracle(name, cs, y, host, flops, threads):
    """CPU half of one row: the fp64 oracle on all host cores (full evaluation, timed) or on
    sampled outputs, the GPU result's normalised errors against it, and the single-threaded
    full evaluation for the smallest workloads."""
    import numpy as np
    import oracle
    x, w, b = host
    bias = b if cs.has_bias else None
    out = {}
    if name in ORACLE_FULL:
        t0 = time.perf_counter()
        y_ref, a_ref = oracle.conv2d(x, w, bias, cs.stride, cs.pad, cs.dil, cs.groups, nthreads=threads)
        dt = time.perf_counter() - t0
        lit, pt = oracle.normalised_errors(y, y_ref, a_ref)
        out["oracle"] = {"kind": "oracle", "sample": "every output", "cores": threads, "seconds": dt,
                         "tflops": flops / dt / 1e12}
        if name in ORACLE_SINGLE_THREAD:
            t0 = time.perf_counter()
            oracle.conv2d(x, w, bias, cs.stride, cs.pad, cs.dil, cs.groups, nthreads=1, want_abs=False)
            dt1 = time.perf_counter() - t0
            out["oracle_single_thread"] = {"cores": 1, "seconds": dt1, "tflops": flops / dt1 / 1e12}
        sample = "every output"
    else:
        rng = np.random.default_rng(12345)
        npts = min(65536, y.size)
        flat = rng.choice(y.size, size=npts, replace=False)
        idx = np.stack(np.unravel_index(flat, y.shape), axis=1).astype(np.int64)
        y_ref, a_ref = oracle.conv2d_points(x, w, bias, idx, cs.stride, cs.pad, cs.dil, cs.groups,
                                            nthreads=threads)
        lit, pt = oracle.normalised_errors(y[tuple(idx.T)], y_ref, a_ref)
        sample = f"{npts} sampled outputs"
    gate = 1e-5 if cs.x_dtype == "f32" else 1e-2
    out["parity"] = {"sample": sample, "err_per_point": pt, "err_literal": lit, "gate": gate, "pass": pt <= gate}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10,
                    help="untimed steps before the timed ones (after the fixed-time clock ramp)")
    ap.add_argument("--ramp-seconds", type=float, default=1.0,
                    help="back-to-back calls for this long before the warm-up: the GPU clocks need "
                         "sustained load to come up")
    ap.add_argument("--workload", default="cfg2")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-per-config", action="store_true", help="skip the per-shape rows")
    ap.add_argument("--no-pack-probe", action="store_true",
                    help="skip the pack probe (its loader-only launches share the microkernel's name, so "
                         "profiling runs leave them out)")
    ap.add_argument("--cold-runs", type=int, default=20)
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (reference kernel for HBM byte counters)")
    ap.add_argument("--summarize-profiles", metavar="DIR",
                    help="write the text summary of rocprofv3 outputs in DIR (no GPU needed) and exit")
    ap.add_argument("--traffic-kernel", default=None,
                    help="with --summarize-profiles: kernel whose traffic goes to profiles/traffic.json")
    ap.add_argument("--sweep", metavar="REPORT",
                    help="time the 500-convolution sweep, write per-convolution rows to REPORT and exit")
    args = ap.parse_args()
    if args.summarize_profiles:
        text, traffic = summarize_profiles(args.summarize_profiles, args.workload)
        print(text)
        if args.traffic_kernel:
            key = [k for k in traffic if args.traffic_kernel in k]
            if len(key) != 1:
                sys.exit(f"traffic kernel {args.traffic_kernel!r} matches {key}")
            try:
                with open(TRAFFIC_FILE) as f:
                    data = json.load(f)
            except (OSError, ValueError):
                data = {}
            # the bench line of the traced run (the profiler's own messages may follow it)
            algo_name = None
            with open(os.path.join(args.summarize_profiles, "bench.json")) as f:
                for line in f:
                    try:
                        algo_name = json.loads(line)["config"]["algo"]
                    except (ValueError, KeyError, TypeError):
                        pass
            if algo_name is None:
                sys.exit(f"no bench line in {args.summarize_profiles}/bench.json")
            data[f"{args.workload}:{algo_name}"] = {
                "kernel": key[0], "bytes_per_launch": traffic[key[0]],
                "kernel_hash": kernel_hash(algo_name)}
            with open(TRAFFIC_FILE, "w") as f:
                json.dump(data, f, indent=1)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the conv2d library runs on a single MI355X)", file=sys.stderr)
        sys.exit(2)

    import torch
    import datagen
    from paper_2407_10730_amd import binding as B
    from paper_2407_10730_amd.runner import DeviceConv

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    B.load()
    if args.sweep:
        print(json.dumps(run_sweep(args.sweep, B, torch)), flush=True)
        return
    cs = datagen.CONFIGS[args.workload]
    print(f"[bench] workload {args.workload}: {describe(cs)}", file=sys.stderr, flush=True)
    dc = DeviceConv(cs)
    nkhw = dc.out_nkhw
    n, k, ho, wo = nkhw
    flops = 2 * n * k * (cs.c // cs.groups) * cs.r * cs.s * ho * wo
    algo = dc.plan(B.CONV2D_ALGO_AUTO).algo
    algo_name = B.ALGO_NAMES[algo]
    plan = dc.plan(algo)

    # headline: the clock ramp, the warm-up, then exactly `steps` calls with no events between
    # kernels (an event pair on the stream around all of them)
    ramp = clock_ramp(dc, algo, args.ramp_seconds, torch)
    wall, ev_ms, _ = time_algo(dc, algo, args.steps, args.warmup, B, torch, B.CONV2D_TIMING_OFF)
    ms_per_step = wall * 1e3 / args.steps
    tflops = flops / (ms_per_step * 1e-3) / 1e12
    kern_ms, kern_src = kernel_duration(dc, algo, ev_ms, B, torch)
    # the breakdown: the same loop with an event pair around every phase launch
    wall_ph, _, bd = time_algo(dc, algo, args.steps, 2, B, torch, B.CONV2D_TIMING_PHASES)
    print(f"[bench] {algo_name}: {ms_per_step*1e3:.1f} us/step (events {ev_ms*1e3:.1f}), {tflops:.1f} TFLOP/s, "
          f"kernel {kern_ms*1e3 if kern_ms else float('nan'):.1f} us ({kern_src})", file=sys.stderr, flush=True)
    y_gpu = dc.y_nchw()

    xdt = cs.x_dtype
    roof = roofline(cs, nkhw, flops, kern_ms)
    roof["kernel"] = f"{algo_name} microkernel ({kernel_label(plan, B)})"
    roof["kernel_us_per_launch"] = None if kern_ms is None else kern_ms * 1e3
    roof["kernel_source"] = kern_src
    roof["traffic"] = load_traffic(args.workload, algo_name)

    # explicit im2col baseline on the same workload: pack-phase share
    ne = max(5, args.steps // 5)
    wall_e, _, _ = time_algo(dc, B.CONV2D_ALGO_IM2COL_GEMM, ne, 3, B, torch, B.CONV2D_TIMING_OFF)
    _, _, bd_e = time_algo(dc, B.CONV2D_ALGO_IM2COL_GEMM, ne, 1, B, torch, B.CONV2D_TIMING_PHASES)
    ms_e = wall_e * 1e3 / ne
    opsum = bd_e["ms"]["in_packing"] + bd_e["ms"]["in_microkernel"] + bd_e["ms"]["in_unpacking"]
    explicit = {
        "ms_per_step": ms_e,
        "tflops": flops / (ms_e * 1e-3) / 1e12,
        "phase_ms_per_step": {p: v / bd_e["fwd_calls"] for p, v in bd_e["ms"].items() if p != "pre_analysis"},
        "pack_share": bd_e["ms"]["in_packing"] / opsum if opsum > 0 else None,
        "t_explicit_over_t_implicit": ms_e / ms_per_step,
    }
    # Winograd on the same workload when it applies (3x3, stride 1)
    wino = None
    if algo != B.CONV2D_ALGO_WINOGRAD:
        try:
            dc.plan(B.CONV2D_ALGO_WINOGRAD)
            wino_ok = True
        except B.Conv2dError:
            wino_ok = False
        if wino_ok:
            wall_w, _, _ = time_algo(dc, B.CONV2D_ALGO_WINOGRAD, ne, 3, B, torch, B.CONV2D_TIMING_OFF)
            _, _, bd_w = time_algo(dc, B.CONV2D_ALGO_WINOGRAD, ne, 1, B, torch, B.CONV2D_TIMING_PHASES)
            ms_w = wall_w * 1e3 / ne
            wino = {"ms_per_step": ms_w, "tflops": flops / (ms_w * 1e-3) / 1e12,
                    "phase_ms_per_step": {p: v / bd_w["fwd_calls"] for p, v in bd_w["ms"].items()
                                          if p != "pre_analysis"},
                    "t_winograd_over_t_main": ms_w / ms_per_step}
    cold = cold_median(dc, algo, args.cold_runs, B, torch)
    # pack probe: the implicit microkernel's loader alone (gather into LDS, no MFMA, no
    # output) against the full microkernel -- an estimate of the fused packing share
    probe = None
    if algo == B.CONV2D_ALGO_IMPLICIT_GEMM and not args.no_pack_probe and kern_ms:
        stream = torch.cuda.current_stream()
        dc.run(algo, stream)
        probe_ms = time_launches(lambda: B.conv2d_pack_probe(dc.desc, dc.x, dc.w, stream), 20, torch)
        probe = {"kind": "estimate (loader-only microkernel / microkernel)",
                 "loader_only_us": probe_ms * 1e3, "microkernel_us": kern_ms * 1e3,
                 "share_estimate": probe_ms / kern_ms}
    peaks = measured_peaks(B, torch)

    out = {
        "metric": METRIC,
        "value": tflops,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"f32": "f32", "bf16": "bf16"}[xdt],
        "data": "synthetic (seeded U[-1,1])",
        "config": {"workload": f"{args.workload}: {describe(cs)}", "algo": algo_name,
                   "flops": flops, "arith_intensity": roof["arith_intensity"]},
        "roofline": roof,
        "kernel_le_step": None if kern_ms is None else kern_ms <= max(ms_per_step, ev_ms) * 1.02,
        "event_ms_per_step": ev_ms,
        "clock_ramp": ramp,
        "breakdown_ms_per_step": {p: v / bd["fwd_calls"] for p, v in bd["ms"].items()
                                  if p != "pre_analysis"},
        "phase_events_overhead_ms_per_step": (wall_ph - wall) * 1e3 / args.steps,
        "fused_phases": bd["fused"],
        "pre_analysis_ms_once": bd["ms"]["pre_analysis"],
        "explicit_im2col": explicit,
        "winograd": wino,
        "cold_cache_ms_median": cold,
        "cold_cache_tflops": flops / (cold * 1e-3) / 1e12,
        "implicit_pack_probe": probe,
        "measured_peaks": peaks,
    }
    if out["kernel_le_step"] is False:
        print("[bench] WARNING: kernel duration exceeds the step time", file=sys.stderr, flush=True)
    host = (dc.x_host, dc.w_host, dc.b_host)
    dc.close()

    # per-shape rows: every GPU measurement first (the host work in between would let the
    # clocks drop), then the oracle on the host cores
    per_gpu = []
    if not args.no_per_config:
        for name in PER_CONFIG:
            if name == args.workload:
                continue
            per_gpu.append((name,) + config_gpu(name, args, B, torch))

    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or len(os.sched_getaffinity(0))
    threads = max(1, min(threads, len(os.sched_getaffinity(0))))
    if not args.no_cpu:
        cb, parity = cpu_baseline(cs, host[0], host[1], host[2], y_gpu, flops // n)
        out["cpu_baseline"] = cb
        cb["gpu_over_oracle"] = out["value"] / cb["value"]
        out["cpu_im2col_gemm_context"], _ = cpu_im2col_gemm(cs, host[0], host[1], host[2], flops // n,
                                                            n_img=min(cs.n, 4))
        out["parity_on_cpu_sample"] = parity
    if per_gpu:
        per = {}
        head_row = {"workload": describe(cs), "algo": algo_name, "steps": args.steps, "ms_per_step": ms_per_step,
                    "event_ms_per_step": ev_ms, "tflops": tflops,
                    "roofline": {kk: roof[kk] for kk in ("bound", "achieved", "peak", "unit", "frac")}
                    | {"kernel_us": roof["kernel_us_per_launch"], "kernel_source": kern_src},
                    "kernel_le_step": out["kernel_le_step"],
                    "explicit_im2col": {"ms_per_step": ms_e, "pack_share": explicit["pack_share"],
                                        "t_explicit_over_t_main": ms_e / ms_per_step}}
        if not args.no_cpu:
            head_row.update(config_oracle(args.workload, cs, y_gpu, host, flops, threads))
        per[args.workload] = head_row
        for name, row, (ccs, y, chost, cflops) in per_gpu:
            if not args.no_cpu:
                row.update(config_oracle(name, ccs, y, chost, cflops, threads))
            per[name] = row
        out["per_config"] = {kk: per[kk] for kk in PER_CONFIG if kk in per}
    if args.calibrate_copy:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(3)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = 1 << 30
        del src, dst
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
