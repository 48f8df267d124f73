"""bench.py's host-side parts: the CPU oracle baseline and the one-GPU guard (no GPU needed)."""
import os
import subprocess
import sys

import numpy as np

import bench
import datagen
import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_cpu_baseline_fields():
    cs = datagen.CONFIGS["cfg1"]
    x, w, b = datagen.make_inputs(cs, "random")
    y, _ = oracle.conv2d(x, w, b, cs.stride, cs.pad, cs.dil, cs.groups)
    flops_per_image = 2 * 16 * 3 * 9 * 32 * 32
    res, parity = bench.cpu_baseline(cs, x, w, b, y.astype(np.float32), flops_per_image, target_s=0.05)
    assert res["kind"] == "oracle" and res["unit"] == "TFLOP/s" and res["value"] > 0
    assert 1 <= res["cores"] <= len(os.sched_getaffinity(0))
    assert res["single_thread"]["cores"] == 1 and res["single_thread"]["value"] > 0
    assert parity["images"] == 1 and parity["err_per_point"] <= 1e-6


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_cpu_im2col_gemm_context_matches_oracle():
    # the host im2col + GEMM context computes the same convolution (checked on a strided,
    # dilated, grouped shape against the oracle)
    cs = datagen.ConvShape(n=2, c=6, h=11, w=9, k=4, r=3, s=2, stride=(2, 1), pad=(1, 1), dil=(2, 1), groups=2,
                           seed=5, has_bias=True)
    x, w, b = datagen.make_inputs(cs, "random")
    y_ref, a_ref = oracle.conv2d(x, w, b, cs.stride, cs.pad, cs.dil, cs.groups)
    res, y = bench.cpu_im2col_gemm(cs, x, w, b, 1.0, n_img=2)
    assert res["value"] > 0 and res["sample"].startswith("first 2")
    assert y.shape == y_ref.shape
    assert oracle.normalised_errors(y, y_ref, a_ref)[1] <= 1e-5
