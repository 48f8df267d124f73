"""The ConvBench-style harness on the GPU: main, baseline and the correctness check of
main against baseline over a small operation list, both results checked against the
oracle through the harness's dumps, and the speedup report on the results."""
import csv
import os
import subprocess

import numpy as np
import pytest

import oracle
from paper_2407_10730_amd import binding as B
from paper_2407_10730_amd import convbench_report as R

pytestmark = pytest.mark.gpu
HARNESS = os.path.join(os.path.dirname(B.__file__), "convbench")

OPS = [
    # name, n, c, h, w, k, r, s, stride, pad, dil, groups, bias, dtype, layout
    ("reg3x3", 2, 32, 17, 15, 48, 3, 3, 1, 1, 1, 1, 1, "f32", "nchw"),
    ("dw", 2, 64, 14, 14, 64, 3, 3, 1, 1, 1, 64, 1, "f32", "nchw"),
    ("pw_s2", 1, 64, 20, 20, 96, 1, 1, 2, 0, 1, 1, 0, "bf16", "nhwc"),
    ("grp_dil", 1, 16, 23, 19, 24, 5, 3, 2, 2, 2, 2, 1, "f32", "nchw"),
    ("stem", 1, 3, 64, 64, 16, 7, 7, 2, 3, 1, 1, 1, "bf16", "nchw"),
]


@pytest.fixture(scope="module")
def ops_csv(tmp_path_factory):
    import torch
    if torch.cuda.device_count() < 1:
        pytest.skip("no GPU")
    p = tmp_path_factory.mktemp("cb") / "ops.csv"
    with open(p, "w") as f:
        f.write(",".join(R.COLUMNS) + "\n")
        for name, n, c, h, w, k, r, s, st, pd, dl, g, b, dt, lay in OPS:
            f.write(f"{name},{n},{c},{h},{w},{k},{r},{s},{st},{st},{pd},{pd},{dl},{dl},{g},{b},{dt},{lay}\n")
    return p


def _run(ops, out, *args):
    print(f"\n[case] convbench {' '.join(args)}", flush=True)
    r = subprocess.run([HARNESS, "--csv", str(ops), "--out", str(out), *args], capture_output=True, text=True,
                       timeout=240)
    with open(out) as f:
        return r, list(csv.DictReader(f))


GATE = {"f32": 1e-5, "bf16": 1e-2}


def test_correctness_main_against_baseline_and_oracle(ops_csv, tmp_path):
    """Correctness mode passes its own main-against-baseline gate, and both of its results, read
    back from the dump with the inputs the GPU read, pass the oracle's per-output gate; the
    harness's per-point error agrees with the one the oracle's denominator gives."""
    for datagen in ("random", "constant"):
        dump = tmp_path / f"dump_{datagen}"
        dump.mkdir()
        r, rows = _run(ops_csv, tmp_path / "c.csv", "--exec", "correctness", "--datagen", datagen,
                       "--dump", str(dump))
        assert r.returncode == 0, r.stderr
        assert [x["name"] for x in rows] == [o[0] for o in OPS]
        for i, (x, op) in enumerate(zip(rows, OPS)):
            assert x["status"] == "ok" and x["correct"] == "1", x
            name, n, c, h, w, k, rr, ss, st, pd, dl, g, b, dt, lay = op
            ho, wo = int(x["ho"]), int(x["wo"])
            hx = np.fromfile(dump / f"{i}.x", dtype=np.float32)
            hx = hx.reshape(n, h, w, c).transpose(0, 3, 1, 2) if lay == "nhwc" else hx.reshape(n, c, h, w)
            hw = np.fromfile(dump / f"{i}.w", dtype=np.float32).reshape(k, c // g, rr, ss)
            hb = np.fromfile(dump / f"{i}.b", dtype=np.float32)
            y_ref, a_ref = oracle.conv2d(hx, hw, hb if b else None, (st, st), (pd, pd), (dl, dl), g)
            ys = {}
            for which in ("y_main", "y_base"):
                y = np.fromfile(dump / f"{i}.{which}", dtype=np.float32)
                y = y.reshape(n, ho, wo, k).transpose(0, 3, 1, 2) if lay == "nhwc" else y.reshape(n, k, ho, wo)
                _, pt = oracle.normalised_errors(y, y_ref, a_ref)
                assert pt <= max(GATE[dt], 2.0 ** -8 if dt == "bf16" else 0), (name, datagen, which, pt)
                ys[which] = y.astype(np.float64)
            e = np.abs(ys["y_main"] - ys["y_base"])
            pos = a_ref > 0
            pt_py = float((e[pos] / a_ref[pos]).max()) if pos.any() else 0.0
            pt_cb = float(x["err_per_point"])
            # the harness's denominator is the library's own |x|*|w| convolution (rounded to the
            # output type), so the two readings agree up to that rounding
            assert pt_cb <= pt_py * 1.02 + 1e-12 and pt_py <= pt_cb * 1.02 + 1e-12, (name, pt_cb, pt_py)


def test_main_and_baseline_timings_and_speedup(ops_csv, tmp_path):
    res = {}
    for exe in ("main", "baseline"):
        r, rows = _run(ops_csv, tmp_path / f"{exe}.csv", "--exec", exe, "--warmups", "2", "--runs", "5")
        assert r.returncode == 0, r.stderr
        for x in rows:
            assert x["status"] == "ok", x
            assert float(x["op_ms"]) > 0 and float(x["tflops"]) > 0
            assert float(x["in_microkernel_ms"]) > 0 and float(x["in_microkernel_calls"]) >= 1
            if exe == "baseline":
                assert x["algo"] == "im2col_gemm" and float(x["in_packing_ms"]) > 0
        res[exe] = rows
    assert {x["algo"] for x in res["main"]} <= {"implicit_gemm", "direct"}
    s = R.speedup(str(tmp_path / "main.csv"), str(tmp_path / "baseline.csv"), str(tmp_path / "s.csv"),
                  str(tmp_path / "plots"))
    assert s["ops"] == len(OPS)
    assert os.path.exists(tmp_path / "plots" / "speedup.png")
