"""The ConvBench-style harness on the CPU: operation lists and their filters, the
executable's planning pass and argument checks, and the speedup report."""
import csv
import os
import subprocess

import pytest

from paper_2407_10730_amd import binding as B
from paper_2407_10730_amd import convbench_report as R
from paper_2407_10730_amd.runner import params_for
import datagen

HARNESS = os.path.join(os.path.dirname(B.__file__), "convbench")


def _rows(path):
    with open(path) as f:
        return list(csv.DictReader(f))


def test_export_configs_and_filters(tmp_path):
    p = tmp_path / "ops.csv"
    assert R.export("configs", str(p), []) == len(datagen.CONFIGS)
    rows = _rows(p)
    assert [r["name"] for r in rows] == list(datagen.CONFIGS)
    assert list(rows[0].keys()) == R.COLUMNS
    grouped = {"dw", "dw_bf16", "grp_g64", "grp_g32"}
    assert R.export("configs", str(p), ["no-grouped"]) == len(datagen.CONFIGS) - len(grouped)
    assert {r["name"] for r in _rows(p)} == set(datagen.CONFIGS) - grouped
    R.export("configs", str(p), ["pointwise"])
    assert {r["name"] for r in _rows(p)} == {"cfg3a", "cfg3b"}
    R.export("configs", str(p), ["bf16"])
    assert {r["name"] for r in _rows(p)} == {"cfg4_bf16", "dw_bf16", "bf16_3x3"}
    R.export("configs", str(p), ["regular", "no-strided", "f32"])
    assert {r["name"] for r in _rows(p)} == {"cfg1", "cfg2"}
    with pytest.raises(ValueError):
        R.export("configs", str(p), ["no-such-filter"])


def test_export_sweep_filtered(tmp_path):
    p = tmp_path / "ops.csv"
    n = R.export("sweep", str(p), ["no-grouped", "no-dilated", "f32"], max_gflop=50.0)
    rows = _rows(p)
    assert 0 < n == len(rows) < 250
    for r in rows:
        assert r["groups"] == "1" and r["dil_h"] == "1" and r["dtype"] == "f32"


def test_harness_dry_run_plans_every_op(tmp_path):
    ops = tmp_path / "ops.csv"
    R.export("configs", str(ops), [])
    out = tmp_path / "res.csv"
    for exe, algo in (("main", B.CONV2D_ALGO_AUTO), ("baseline", B.CONV2D_ALGO_IM2COL_GEMM)):
        r = subprocess.run([HARNESS, "--csv", str(ops), "--out", str(out), "--exec", exe, "--dry-run"],
                           capture_output=True, text=True, timeout=60)
        assert r.returncode == 0, r.stderr
        res = _rows(out)
        assert [x["name"] for x in res] == list(datagen.CONFIGS)
        for x in res:
            cs = datagen.CONFIGS[x["name"]]
            d = B.conv2d_desc_create(params_for(cs))
            try:
                plan = B.conv2d_plan_query(d, algo)
                ho, wo = B.conv2d_output_shape(d)[2:]
            finally:
                B.conv2d_desc_destroy(d)
            assert x["status"] == "ok"
            assert x["algo"] == B.ALGO_NAMES[plan.algo]
            assert (int(x["ho"]), int(x["wo"])) == (ho, wo)
            assert (int(x["tile_m"]), int(x["tile_n"])) == (plan.tile_m, plan.tile_n)


# (name, n, c, h, w, k, r, s, stride, pad, dil, groups, bias, dtype, layout)
DATA_OPS = [
    ("f32", 2, 5, 7, 6, 4, 3, 3, 1, 1, 1, 1, 1, "f32", "nchw"),
    ("bf16_nhwc", 1, 8, 5, 9, 6, 3, 1, 2, 1, 1, 2, 1, "bf16", "nhwc"),
    ("nobias", 3, 4, 4, 4, 3, 1, 1, 1, 0, 1, 1, 0, "f32", "nhwc"),
]


def _ops_file(path, ops):
    with open(path, "w") as f:
        f.write(",".join(R.COLUMNS) + "\n")
        for name, n, c, h, w, k, r, s, st, pd, dl, g, b, dt, lay in ops:
            f.write(f"{name},{n},{c},{h},{w},{k},{r},{s},{st},{st},{pd},{pd},{dl},{dl},{g},{b},{dt},{lay}\n")


@pytest.mark.parametrize("mode", ["random", "constant"])
def test_harness_data_is_the_datagen_streams(tmp_path, mode):
    """The harness draws operation i's data from the same SplitMix64 streams as datagen (seed
    S + i, tensors x / w / bias), bit for bit, rounds bf16 operations' values the same way, and
    lays x out in the operation's layout; the dump holds exactly what the GPU reads."""
    import numpy as np
    ops = tmp_path / "ops.csv"
    _ops_file(ops, DATA_OPS)
    dump = tmp_path / "dump"
    dump.mkdir()
    r = subprocess.run([HARNESS, "--csv", str(ops), "--out", str(tmp_path / "o.csv"), "--dry-run", "--seed", "4242",
                        "--datagen", mode, "--dump", str(dump)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    for i, (name, n, c, h, w, k, rr, ss, st, pd, dl, g, b, dt, lay) in enumerate(DATA_OPS):
        cs = datagen.ConvShape(n=n, c=c, h=h, w=w, k=k, r=rr, s=ss, stride=(st, st), pad=(pd, pd), dil=(dl, dl),
                               groups=g, has_bias=bool(b), x_dtype=dt, y_dtype=dt, seed=4242 + i)
        x, wt, bias = datagen.make_inputs(cs, mode, const=(0.5, 0.25, 1.0))
        hx = np.fromfile(dump / f"{i}.x", dtype=np.float32)
        if lay == "nhwc":
            hx = hx.reshape(n, h, w, c).transpose(0, 3, 1, 2)
        assert np.array_equal(hx.reshape(x.shape).view(np.uint32), x.view(np.uint32)), name
        assert np.array_equal(np.fromfile(dump / f"{i}.w", dtype=np.float32).reshape(wt.shape).view(np.uint32),
                              wt.view(np.uint32)), name
        assert np.array_equal(np.fromfile(dump / f"{i}.b", dtype=np.float32).view(np.uint32), bias.view(np.uint32)), name


def test_harness_rejects_bad_input(tmp_path):
    bad = tmp_path / "bad.csv"
    bad.write_text("name,n,c\nx,1,2\n")
    r = subprocess.run([HARNESS, "--csv", str(bad), "--out", str(tmp_path / "o.csv")], capture_output=True,
                       text=True, timeout=60)
    assert r.returncode == 2 and "missing column" in r.stderr
    ops = tmp_path / "ops.csv"
    R.export("configs", str(ops), [])
    for args in (["--exec", "fast"], ["--datagen", "zeros"], ["--runs", "0"], ["--bogus"]):
        r = subprocess.run([HARNESS, "--csv", str(ops), "--out", str(tmp_path / "o.csv"), *args],
                           capture_output=True, text=True, timeout=60)
        assert r.returncode == 2, args
    # an operation the library rejects is reported in its row, and the exit status says so
    odd = tmp_path / "odd.csv"
    odd.write_text(",".join(R.COLUMNS) + "\nsmall,1,3,2,2,16,5,5,1,1,0,0,1,1,1,1,f32,nchw\n")
    r = subprocess.run([HARNESS, "--csv", str(odd), "--out", str(tmp_path / "o.csv"), "--dry-run"],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 1
    assert _rows(tmp_path / "o.csv")[0]["status"] != "ok"


def _result_file(path, times):
    cols = ["name", "status", "algo", "op_ms"] + [f"{p}_ms" for p in R.PHASES]
    with open(path, "w", newline="") as f:
        wr = csv.DictWriter(f, fieldnames=cols)
        wr.writeheader()
        for name, (op, pack, mk) in times.items():
            row = {c: 0.0 for c in cols}
            row.update({"name": name, "status": "ok", "algo": "x", "op_ms": op, "in_packing_ms": pack,
                        "in_microkernel_ms": mk})
            wr.writerow(row)


def test_speedup_report(tmp_path):
    _result_file(tmp_path / "m.csv", {"a": (1.0, 0.0, 1.0), "b": (2.0, 0.0, 2.0), "c": (4.0, 0.0, 4.0)})
    _result_file(tmp_path / "b.csv", {"a": (2.0, 1.0, 1.0), "b": (1.0, 0.25, 0.75), "c": (8.0, 4.0, 4.0)})
    s = R.speedup(str(tmp_path / "m.csv"), str(tmp_path / "b.csv"), str(tmp_path / "s.csv"), str(tmp_path / "plots"))
    assert s["ops"] == 3
    assert s["main_faster_share"] == pytest.approx(2 / 3)
    assert s["geomean_speedup"] == pytest.approx((2.0 * 0.5 * 2.0) ** (1 / 3))
    rows = {r["name"]: r for r in _rows(tmp_path / "s.csv")}
    assert float(rows["b"]["speedup"]) == pytest.approx(0.5)
    assert float(rows["c"]["baseline_pack_share"]) == pytest.approx(0.5)
    assert os.path.exists(tmp_path / "plots" / "speedup.png")
    assert os.path.exists(tmp_path / "plots" / "breakdown.png")
