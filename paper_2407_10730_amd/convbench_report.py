"""Operation lists and reports for the ConvBench-style harness (`convbench` executable).

The paper's workflow (Sec. III-B, III-C): a set of convolution operations is filtered to
what an implementation supports and exported to CSV; the harness runs the main and the
baseline implementation over that CSV and writes measured times and call counts; a script
then computes the main-over-baseline speedup per operation and draws speedup and
time-breakdown plots.  The paper's operation set (harvested from model zoos) is not
available here, so the operation lists are the fixed workloads and the seeded sweep of
this library's generator.

  python -m paper_2407_10730_amd.convbench_report export --set sweep --out ops.csv \\
         [--filter no-grouped,no-dilated,...] [--max-gflop X]
  python -m paper_2407_10730_amd.convbench_report speedup --main main.csv --baseline base.csv \\
         --out speedup.csv [--plots DIR]

Filters: no-grouped, no-dilated, no-strided, pointwise, regular (not pointwise, not grouped),
f32, bf16.
"""
import argparse
import csv
import math
import os
import sys

COLUMNS = ["name", "n", "c", "h", "w", "k", "r", "s", "stride_h", "stride_w", "pad_h", "pad_w", "dil_h", "dil_w",
           "groups", "bias", "dtype", "layout"]
PHASES = ["pre_analysis", "pre_reorder", "in_tiling", "in_packing", "in_microkernel", "in_unpacking", "post_reorder"]
FILTERS = ("no-grouped", "no-dilated", "no-strided", "pointwise", "regular", "f32", "bf16")


def op_row(cs):
    return {"name": cs.name, "n": cs.n, "c": cs.c, "h": cs.h, "w": cs.w, "k": cs.k, "r": cs.r, "s": cs.s,
            "stride_h": cs.stride[0], "stride_w": cs.stride[1], "pad_h": cs.pad[0], "pad_w": cs.pad[1],
            "dil_h": cs.dil[0], "dil_w": cs.dil[1], "groups": cs.groups, "bias": int(cs.has_bias),
            "dtype": cs.x_dtype, "layout": cs.layout}


def keep(row, filters):
    """The filtering mechanism: True when the operation passes every filter."""
    g, r, s = int(row["groups"]), int(row["r"]), int(row["s"])
    pointwise = r == 1 and s == 1
    for f in filters:
        if f == "no-grouped" and g > 1:
            return False
        if f == "no-dilated" and (int(row["dil_h"]) > 1 or int(row["dil_w"]) > 1):
            return False
        if f == "no-strided" and (int(row["stride_h"]) > 1 or int(row["stride_w"]) > 1):
            return False
        if f == "pointwise" and not pointwise:
            return False
        if f == "regular" and (pointwise or g > 1):
            return False
        if f in ("f32", "bf16") and row["dtype"] != f:
            return False
    return True


def gflop(row, ho, wo):
    return 2.0 * int(row["n"]) * int(row["k"]) * (int(row["c"]) // int(row["groups"])) * int(row["r"]) * \
        int(row["s"]) * ho * wo / 1e9


def export(which, path, filters, max_gflop=None):
    """Write the operation list `which` ("configs" or "sweep") as CSV; returns the row count."""
    import datagen
    from paper_2407_10730_amd import binding as B
    from paper_2407_10730_amd.runner import params_for

    def out_hw(cs):
        d = B.conv2d_desc_create(params_for(cs))
        try:
            return B.conv2d_output_shape(d)[2:]
        finally:
            B.conv2d_desc_destroy(d)

    bad = [f for f in filters if f not in FILTERS]
    if bad:
        raise ValueError(f"unknown filters {bad}; known: {', '.join(FILTERS)}")
    if which == "configs":
        shapes = [cs.with_(name=name) for name, cs in datagen.CONFIGS.items()]
    elif which == "sweep":
        shapes, _ = datagen.sweep_shapes(out_hw)
    else:
        raise ValueError(which)
    rows = []
    for cs in shapes:
        row = op_row(cs)
        if not keep(row, filters):
            continue
        if max_gflop is not None and gflop(row, *out_hw(cs)) > max_gflop:
            continue
        rows.append(row)
    with open(path, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=COLUMNS)
        wr.writeheader()
        wr.writerows(rows)
    return len(rows)


def read_results(path):
    with open(path) as f:
        return list(csv.DictReader(f))


def speedup(main_path, base_path, out_path, plots=None):
    """Join the main and baseline result files by operation name: speedup = baseline
    Operation Time / main Operation Time.  Returns a summary dict."""
    main = {r["name"]: r for r in read_results(main_path) if r["status"] == "ok"}
    base = {r["name"]: r for r in read_results(base_path) if r["status"] == "ok"}
    names = [n for n in main if n in base and float(main[n]["op_ms"]) > 0 and float(base[n]["op_ms"]) > 0]
    rows = []
    for n in names:
        m, b = main[n], base[n]
        tm, tb = float(m["op_ms"]), float(b["op_ms"])
        conv_m = sum(float(m[f"{p}_ms"]) for p in PHASES[2:6])
        conv_b = sum(float(b[f"{p}_ms"]) for p in PHASES[2:6])
        rows.append({"name": n, "main_algo": m["algo"], "baseline_algo": b["algo"], "main_ms": tm,
                     "baseline_ms": tb, "speedup": tb / tm,
                     "main_convolution_ms": conv_m, "baseline_convolution_ms": conv_b,
                     "baseline_pack_share": float(b["in_packing_ms"]) / conv_b if conv_b > 0 else 0.0})
    with open(out_path, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=list(rows[0].keys()) if rows else ["name"])
        wr.writeheader()
        wr.writerows(rows)
    sp = [r["speedup"] for r in rows]
    summary = {"ops": len(rows), "main_faster_share": sum(1 for v in sp if v > 1.0) / len(sp) if sp else None,
               "geomean_speedup": math.exp(sum(math.log(v) for v in sp) / len(sp)) if sp else None,
               "max_speedup": max(sp) if sp else None, "min_speedup": min(sp) if sp else None}
    if plots and rows:
        _plots(rows, main, base, plots)
    return summary


def _plots(rows, main, base, outdir):
    import matplotlib
    matplotlib.use("Agg")
    import matplotlib.pyplot as plt
    os.makedirs(outdir, exist_ok=True)
    rows = sorted(rows, key=lambda r: r["speedup"])
    fig, ax = plt.subplots(figsize=(10, 4))
    ax.plot(range(len(rows)), [r["speedup"] for r in rows], ".")
    ax.axhline(1.0, color="k", lw=0.8)
    ax.set_yscale("log")
    ax.set_xlabel("operation (sorted)")
    ax.set_ylabel("baseline time / main time")
    ax.set_title("main over baseline, per operation")
    fig.tight_layout()
    fig.savefig(os.path.join(outdir, "speedup.png"), dpi=120)
    plt.close(fig)
    # mean time breakdown per phase, main vs baseline
    fig, ax = plt.subplots(figsize=(6, 4))
    bottom = [0.0, 0.0]
    for p in PHASES[1:]:
        vals = [sum(float(main[r["name"]][f"{p}_ms"]) for r in rows) / len(rows),
                sum(float(base[r["name"]][f"{p}_ms"]) for r in rows) / len(rows)]
        ax.bar(["main", "baseline"], vals, bottom=bottom, label=p)
        bottom = [bottom[0] + vals[0], bottom[1] + vals[1]]
    ax.set_ylabel("mean ms per operation")
    ax.set_title("time breakdown by phase")
    ax.legend(fontsize=7)
    fig.tight_layout()
    fig.savefig(os.path.join(outdir, "breakdown.png"), dpi=120)
    plt.close(fig)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    e = sub.add_parser("export", help="write an operation list as CSV")
    e.add_argument("--set", choices=("configs", "sweep"), default="sweep")
    e.add_argument("--out", required=True)
    e.add_argument("--filter", default="", help="comma-separated: " + ", ".join(FILTERS))
    e.add_argument("--max-gflop", type=float, default=None)
    s = sub.add_parser("speedup", help="main over baseline per operation, with plots")
    s.add_argument("--main", required=True)
    s.add_argument("--baseline", required=True)
    s.add_argument("--out", required=True)
    s.add_argument("--plots", default=None)
    a = ap.parse_args(argv)
    if a.cmd == "export":
        n = export(a.set, a.out, [f for f in a.filter.split(",") if f], a.max_gflop)
        print(f"{n} operations written to {a.out}")
    else:
        print(speedup(a.main, a.baseline, a.out, a.plots))
    return 0


if __name__ == "__main__":
    sys.exit(main())
