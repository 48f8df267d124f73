"""conv2d_fwd_noalloc, the entry point that allocates nothing, against conv2d_fwd (needs the GPU).

Each case creates the same operation once, runs conv2d_fwd into one output and
conv2d_fwd_noalloc into another, and requires the two to agree bit for bit (the
same kernels on the same inputs; only where their workspaces live differs), and
the no-allocation result to pass the oracle gate.  Two no-allocation calls run
back to back before either result is read, the second on a smaller input, so the
second overwrites the scratch array the first used.
"""
import os

import numpy as np
import pytest

import datagen
import oracle
from paper_2407_10730_amd import binding as B
from paper_2407_10730_amd.runner import DeviceConv

pytestmark = pytest.mark.gpu

GATE = {"f32": 1e-5, "bf16": 1e-2}
CFG = datagen.CONFIGS


def _shape(**kw):
    base = dict(n=2, c=24, h=20, w=20, k=40, r=3, s=3, pad=(1, 1), seed=77)
    base.update(kw)
    return datagen.ConvShape(**base)


# (first, second, env at descriptor creation): the first input is the larger one
PAIRS = [
    # tiled GEMM with the tail split (partials and counters in the scratch) and the tap-major
    # filter copy, then the sliced kernel
    ("cfg2-then-cfg1", CFG["cfg2"], CFG["cfg1"], {}),
    # the tap-table gather (table written into the scratch by a kernel), then an NHWC
    # operation whose x and y go through reordered copies in the scratch
    ("table-then-nhwc", _shape(n=4, c=24, k=72, h=30, w=30), _shape(layout="nhwc", c=16, k=24),
     {"CONV2D_SLICE": "0"}),
    # split reduction (partials in the scratch), then bf16 with the NHWC copy of x
    ("split-then-bf16", _shape(n=1, c=512, h=7, w=7, k=512, seed=5),
     _shape(n=2, c=64, h=14, w=14, k=64, x_dtype="bf16", y_dtype="bf16", seed=6),
     {"CONV2D_NHWC_GATHER": "1"}),
    # depthwise NHWC (filters reordered into the scratch), then a grouped direct layer
    ("dw-nhwc-then-grouped", _shape(n=4, c=64, k=64, groups=64, layout="nhwc", h=28, w=28),
     _shape(n=2, c=32, k=32, groups=8, h=12, w=12), {}),
]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load()
    yield
    torch.cuda.synchronize()


class _Env:
    def __init__(self, env):
        self.env, self.old = env, {}

    def __enter__(self):
        for k, v in self.env.items():
            self.old[k] = os.environ.get(k)
            os.environ[k] = v

    def __exit__(self, *exc):
        for k, v in self.old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def _noalloc_output(dc):
    import torch
    y = torch.empty_like(dc.y)
    B.conv2d_fwd_noalloc(dc.desc, dc.x, dc.w, dc.b, y, B.CONV2D_ALGO_AUTO, torch.cuda.current_stream())
    return y


def _host(y, cs):
    a = y.float().cpu().numpy().astype(np.float64)
    return np.ascontiguousarray(a.transpose(0, 3, 1, 2)) if cs.layout == "nhwc" else a


@pytest.mark.parametrize("pair", PAIRS, ids=[p[0] for p in PAIRS])
def test_noalloc_matches_fwd_twice(pair):
    import torch
    name, big, small, env = pair
    print(f"\n[case] no-alloc {name}: {big} then {small}", flush=True)
    with _Env(env):
        d1, d2 = DeviceConv(big), DeviceConv(small)
    try:
        y1 = _noalloc_output(d1)
        y2 = _noalloc_output(d2)   # reuses the scratch the first call used
        d1.run()
        d2.run()
        torch.cuda.synchronize()
        for dc, y_na in ((d1, y1), (d2, y2)):
            cs = dc.cs
            assert torch.equal(y_na, dc.y), f"{cs}: no-allocation result differs from conv2d_fwd"
            y_ref, a_ref = oracle.conv2d(dc.x_host, dc.w_host, dc.b_host, cs.stride, cs.pad, cs.dil,
                                         cs.groups)
            _, pt = oracle.normalised_errors(_host(y_na, cs), y_ref, a_ref)
            gate = GATE[cs.x_dtype] if cs.y_dtype == "f32" else max(GATE[cs.x_dtype], 2.0 ** -8)
            assert pt <= gate, f"{cs}: per-point error {pt:.3e}"
        # and once more in the other order (the smaller operation first)
        y2b = _noalloc_output(d2)
        y1b = _noalloc_output(d1)
        torch.cuda.synchronize()
        assert torch.equal(y1b, d1.y) and torch.equal(y2b, d2.y)
    finally:
        d1.close()
        d2.close()


def test_noalloc_rejects_what_does_not_fit():
    """The explicit path of the 3x3 workload needs a 231 MB column matrix: E_SCRATCH, and
    conv2d_fwd still runs it."""
    import torch
    dc = DeviceConv(CFG["cfg2"])
    try:
        with pytest.raises(B.Conv2dError) as ei:
            B.conv2d_fwd_noalloc(dc.desc, dc.x, dc.w, dc.b, dc.y, B.CONV2D_ALGO_IM2COL_GEMM,
                                 torch.cuda.current_stream())
        assert ei.value.status == B.CONV2D_E_SCRATCH
        dc.run(B.CONV2D_ALGO_IM2COL_GEMM)
        torch.cuda.synchronize()
    finally:
        dc.close()
