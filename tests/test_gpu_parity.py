"""Parity of the HIP conv2d library against the fp64 CPU oracle (needs the GPU).

Gates (per-output normalised error |y - y_ref| / (|b| + sum |x*w|)):
fp32 inputs 1e-5, bf16 inputs 1e-2 (fp32 accumulation; the oracle reads the
same bf16-rounded values).  Integer-valued data (every partial sum exact in
fp32) must match the oracle bit for bit, for every algorithm and dtype.
"""
import os

import numpy as np
import pytest

import datagen
import oracle
from paper_2407_10730_amd import binding as B
from paper_2407_10730_amd.runner import DeviceConv, params_for

pytestmark = pytest.mark.gpu

GATE = {"f32": 1e-5, "bf16": 1e-2}
IMPLICIT, IM2COL, DIRECT = B.CONV2D_ALGO_IMPLICIT_GEMM, B.CONV2D_ALGO_IM2COL_GEMM, B.CONV2D_ALGO_DIRECT
ALGO_IDS = {IMPLICIT: "implicit", IM2COL: "im2col", DIRECT: "direct", B.CONV2D_ALGO_WINOGRAD: "winograd",
            B.CONV2D_ALGO_AUTO: "auto"}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load()
    yield
    torch.cuda.synchronize()


_ORACLE_CACHE = {}


def _reference(cs, mode, inputs):
    key = (cs, mode)
    if key not in _ORACLE_CACHE:
        x, w, b = inputs
        _ORACLE_CACHE[key] = oracle.conv2d(x, w, b if cs.has_bias else None, cs.stride, cs.pad,
                                           cs.dil, cs.groups)
    return _ORACLE_CACHE[key]


class _Kernel:
    """Forces the implicit family's microkernel while descriptors are created: kernel None =
    planner's choice, "0" = tiled GEMM, "1" = sliced kernel (when it fits), "nhwc" = tiled
    GEMM with the bf16 NHWC gather (when C/g allows); waves = the sliced kernel's waves per
    block ("4", "8", or "16" for fp32; None = planner's choice)."""

    def __init__(self, force, waves=None):
        if force == "nhwc":
            self.set = {"CONV2D_SLICE": "0", "CONV2D_NHWC_GATHER": "1", "CONV2D_SLICE_WAVES": None}
        else:
            self.set = {"CONV2D_SLICE": force, "CONV2D_SLICE_WAVES": waves,
                        "CONV2D_NHWC_GATHER": None if force is None else "0"}
        self.old = {}

    def __enter__(self):
        for k, v in self.set.items():
            self.old[k] = os.environ.get(k)
            if v is not None:
                os.environ[k] = v
        return self

    def __exit__(self, *exc):
        for k, v in self.old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def _nhwc_ok(cs):
    """The bf16 NHWC gather takes C/g a multiple of 32, or C/g = 8 or 16."""
    cg = cs.c // cs.groups
    return cs.x_dtype == "bf16" and (cg % 32 == 0 or cg in (8, 16))


def _run(cs, algo, mode="random", kernel=None, waves=None):
    import torch
    print(f"\n[case] {cs} algo={ALGO_IDS[algo]} kernel={kernel} waves={waves} mode={mode}", flush=True)
    with _Kernel(kernel, waves):
        dc = DeviceConv(cs, mode)
    try:
        if kernel == "1" and dc.plan(algo).kernel != B.CONV2D_KERNEL_SLICE:
            pytest.skip("the sliced kernel does not fit this shape")
        if kernel == "nhwc" and not _nhwc_ok(cs):
            pytest.skip("the NHWC gather needs bf16 and C/g a multiple of 32, or 8 or 16")
        dc.run(algo)
        torch.cuda.synchronize()
        y = dc.y_nchw()
    finally:
        dc.close()
    return y, (dc.x_host, dc.w_host, dc.b_host)


def _check(cs, algo, mode="random", kernel=None, waves=None, exact=True):
    """exact=False: integer data checked against the gate instead of bit for bit (an algorithm
    whose intermediate values are not all representable, e.g. Winograd F(4x4, 3x3))."""
    y, inputs = _run(cs, algo, mode, kernel, waves)
    y_ref, a_ref = _reference(cs, mode, inputs)
    assert y.shape == y_ref.shape
    if mode == "integer" and cs.y_dtype == "f32" and exact:
        bad = np.argwhere(y != y_ref)
        assert bad.size == 0, f"{len(bad)} mismatches, first at {bad[0]}: {y[tuple(bad[0])]} vs {y_ref[tuple(bad[0])]}"
        return 0.0
    lit, pt = oracle.normalised_errors(y, y_ref, a_ref)
    gate = GATE[cs.x_dtype]
    if cs.y_dtype == "bf16":
        gate = max(gate, 2.0 ** -8)
    assert pt <= gate, f"per-point error {pt:.3e} > {gate} (literal {lit:.3e})"
    return pt


# ------------------------------------------------------------------ the fixed workloads

FULL = ["cfg1", "cfg2", "cfg3a", "cfg3b", "cfg4", "cfg4_bf16"]


@pytest.mark.parametrize("algo", [IMPLICIT, IM2COL], ids=lambda a: ALGO_IDS[a])
@pytest.mark.parametrize("name", FULL)
def test_config_parity(name, algo):
    _check(datagen.CONFIGS[name], algo)


@pytest.mark.parametrize("kernel", [("0", None), ("1", "4"), ("1", "8"), ("1", "16")],
                         ids=["gemm", "slice4", "slice8", "slice16"])
@pytest.mark.parametrize("name", ["cfg1", "cfg4", "cfg4_bf16"])
def test_config_parity_both_implicit_kernels(name, kernel):
    _check(datagen.CONFIGS[name], IMPLICIT, kernel=kernel[0], waves=kernel[1])
    _check(datagen.CONFIGS[name], IMPLICIT, "integer", kernel=kernel[0], waves=kernel[1])


@pytest.mark.parametrize("algo", [DIRECT, IMPLICIT, IM2COL], ids=lambda a: ALGO_IDS[a])
def test_depthwise_config_parity(algo):
    _check(datagen.CONFIGS["dw"], algo)


@pytest.mark.parametrize("name", ["cfg1", "cfg2", "cfg3b", "cfg4", "dw"])
def test_config_exact_integer(name):
    cs = datagen.CONFIGS[name].with_(w_scale=None)
    algos = [DIRECT] if name == "dw" else [IMPLICIT, IM2COL]
    for algo in algos:
        _check(cs, algo, "integer")
        _check(cs.with_(x_dtype="bf16"), algo, "integer")


# ------------------------------------------------------------------ edge grid

def _shape(n, c, h, w, k, r, s, st=(1, 1), pd=(0, 0), dl=(1, 1), g=1, seed=100, bias=True):
    return datagen.ConvShape(n=n, c=c, h=h, w=w, k=k, r=r, s=s, stride=st, pad=pd, dil=dl, groups=g,
                             seed=seed, has_bias=bias)


EDGE = [
    _shape(1, 3, 5, 7, 5, 3, 3, pd=(1, 1)),
    _shape(2, 5, 11, 9, 7, 5, 3, st=(2, 1), pd=(2, 1), dl=(1, 2)),
    _shape(3, 6, 8, 8, 6, 3, 3, pd=(1, 1), g=6),
    _shape(1, 4, 7, 7, 8, 2, 2, g=2),
    _shape(2, 8, 9, 10, 70, 1, 1),
    _shape(1, 3, 6, 6, 4, 7, 7, pd=(3, 3)),
    _shape(1, 2, 4, 4, 3, 3, 3, st=(3, 3), pd=(3, 3), dl=(2, 2)),
    _shape(2, 64, 14, 14, 130, 3, 3, st=(2, 2), pd=(1, 1)),
    _shape(1, 1, 1, 1, 1, 1, 1),
    _shape(1, 3, 17, 1, 5, 3, 1, pd=(1, 0)),
    _shape(2, 16, 9, 9, 32, 3, 3, pd=(2, 2), dl=(2, 2), g=4),
    _shape(3, 19, 23, 23, 70, 3, 3, pd=(1, 1)),
    _shape(1, 150, 6, 6, 33, 3, 3, pd=(1, 1), bias=False),
    _shape(2, 3, 30, 30, 64, 7, 7, st=(2, 2), pd=(3, 3)),
    _shape(1, 8, 5, 13, 9, 1, 5, st=(1, 3), pd=(0, 2)),
    _shape(4, 12, 7, 7, 12, 3, 3, st=(2, 2), pd=(1, 1), g=12),
    _shape(1, 256, 7, 7, 512, 3, 3, pd=(1, 1)),
    # channel blocks of 16/32 (tap-major gather) with padding, dilation and rectangular filters
    _shape(2, 32, 9, 12, 40, 3, 3, pd=(1, 1)),
    _shape(1, 16, 6, 4, 8, 3, 3, st=(2, 1), pd=(1, 2), dl=(1, 2)),
    _shape(3, 48, 5, 8, 70, 5, 5, pd=(2, 2)),
    _shape(1, 16, 3, 20, 16, 1, 7, pd=(0, 3)),
    # depthwise: multiplier 2, 5x5 dilated, 7x7 stride 2, widths with and without W % 4 == 0,
    # planes taller than one band
    _shape(2, 8, 12, 12, 16, 3, 3, pd=(1, 1), g=8),
    _shape(1, 5, 13, 16, 5, 5, 5, pd=(4, 4), dl=(2, 2), g=5),
    _shape(2, 6, 19, 17, 6, 7, 7, st=(2, 2), pd=(3, 3), g=6),
    _shape(1, 3, 150, 124, 3, 3, 3, st=(1, 2), pd=(1, 1), g=3),
    _shape(3, 4, 7, 7, 4, 1, 1, g=4),
    # depthwise at stride 2 with a 1x1 filter or an even dilation (only even input rows kept),
    # one plane tall enough for several bands
    _shape(2, 6, 15, 16, 6, 1, 1, st=(2, 2), g=6),
    _shape(1, 4, 21, 19, 4, 3, 3, st=(2, 2), pd=(2, 2), dl=(2, 2), g=4),
    _shape(2, 3, 40, 24, 3, 5, 5, st=(2, 2), pd=(4, 4), dl=(2, 2), g=3),
    _shape(1, 2, 300, 40, 2, 3, 3, st=(2, 2), pd=(2, 2), dl=(2, 2), g=2),
]
VARIANTS = [("nchw", "f32", "f32"), ("nhwc", "f32", "f32"), ("nchw", "bf16", "bf16"),
            ("nhwc", "bf16", "f32")]


# bf16 layers the planner sends through the NHWC gather (C/g multiple of 32, high arithmetic
# intensity): stage depths 32 and 64, stride, dilation, padding, groups, NHWC in and out,
# ragged pixel and channel tiles
NHWC_BF16 = [
    _shape(4, 64, 28, 28, 128, 3, 3, pd=(1, 1), seed=210),
    _shape(2, 32, 30, 26, 96, 3, 3, st=(2, 2), pd=(1, 1), seed=211),
    _shape(2, 128, 17, 19, 70, 5, 5, pd=(4, 4), dl=(2, 2), seed=212),
    _shape(1, 256, 14, 14, 256, 3, 3, pd=(1, 1), g=2, seed=213),
    _shape(3, 96, 9, 9, 200, 1, 1, seed=214),
    _shape(2, 64, 23, 23, 64, 7, 7, st=(2, 2), pd=(3, 3), seed=215),
    # C/g = 16 or 8: two or four whole taps per 32-deep stage, the last stage part empty
    _shape(2, 16, 20, 22, 96, 3, 3, pd=(1, 1), seed=216),
    _shape(2, 8, 19, 17, 70, 5, 5, pd=(2, 2), seed=217),
    _shape(1, 32, 15, 15, 64, 3, 3, st=(2, 2), pd=(2, 2), dl=(2, 2), g=2, seed=218),
    _shape(3, 16, 9, 9, 200, 1, 1, seed=219),
    _shape(1, 64, 13, 13, 40, 3, 3, pd=(1, 1), g=8, seed=220),
    # one and three 64-deep stages (the two-set prefetch loop's shortest and odd lengths)
    _shape(2, 64, 11, 13, 72, 1, 1, seed=221),
    _shape(1, 192, 9, 10, 64, 1, 1, pd=(0, 0), seed=222),
]


# pf: register sets of the 64-deep-stage kernels (2, the planner's choice, or 1)
@pytest.mark.parametrize("pf", ["2", "1"])
@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
@pytest.mark.parametrize("idx", range(len(NHWC_BF16)))
def test_bf16_nhwc_gather(idx, layout, pf, monkeypatch):
    monkeypatch.setenv("CONV2D_BF16_PF", pf)
    cs = NHWC_BF16[idx].with_(layout=layout, x_dtype="bf16", y_dtype="bf16")
    with _Kernel("nhwc"):
        dc = DeviceConv(cs, "random")
    try:
        assert dc.plan(IMPLICIT).needs_reorder == 1 or layout == "nhwc"
    finally:
        dc.close()
    _check(cs, IMPLICIT, "random", "nhwc")
    _check(cs.with_(y_dtype="f32"), IMPLICIT, "integer", "nhwc")


# split reductions: layers with few output tiles and long reductions (the planner splits
# them), and forced splits through every gather; partial sums are added in split order
SPLIT = [
    (_shape(1, 512, 7, 7, 256, 3, 3, pd=(1, 1), seed=230), None),
    (_shape(2, 96, 5, 6, 40, 3, 3, pd=(1, 1), seed=231), "5"),
    (_shape(1, 37, 9, 9, 33, 5, 3, st=(2, 1), pd=(2, 1), seed=232), "3"),
    (_shape(1, 64, 12, 12, 70, 3, 3, pd=(2, 2), dl=(2, 2), g=2, seed=233), "4"),
    (_shape(1, 16, 9, 9, 40, 5, 5, pd=(2, 2), seed=234), "3"),
]


@pytest.mark.parametrize("dt", ["f32", "bf16", "bf16-nhwc"])
@pytest.mark.parametrize("idx", range(len(SPLIT)))
def test_split_reduction(idx, dt):
    base, force = SPLIT[idx]
    cs = base.with_(x_dtype="f32" if dt == "f32" else "bf16", y_dtype="f32" if dt == "f32" else "bf16")
    env = {"CONV2D_KSPLIT": force} if force else {}
    kernel = "nhwc" if dt == "bf16-nhwc" else "0"
    old = {k: os.environ.get(k) for k in env}
    os.environ.update(env)
    try:
        with _Kernel(kernel):
            dc = DeviceConv(cs, "random")
        try:
            plan = dc.plan(IMPLICIT)
        finally:
            dc.close()
        if dt == "bf16-nhwc" and not _nhwc_ok(cs):
            pytest.skip("the NHWC gather needs C/g a multiple of 32")
        assert plan.ksplit > 1, plan.ksplit
        _check(cs, IMPLICIT, "random", kernel)
        _check(cs.with_(y_dtype="f32"), IMPLICIT, "integer", kernel)
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


# tail split: the tiles past the last multiple of the CU count are computed in pieces of
# consecutive stages by extra blocks of the launch, and the last piece of a tile to finish adds
# the partials in piece order.  Forced here on small shapes (every tile in pieces) through
# every gather, with ragged channel and pixel tiles; each descriptor runs twice, since the
# arrival counters must be back at zero after a call, and both results must be identical.
TAIL = [
    (_shape(2, 32, 13, 11, 70, 3, 3, pd=(1, 1), seed=240), "3"),
    (_shape(1, 37, 9, 9, 33, 5, 3, st=(2, 1), pd=(2, 1), seed=241), "4"),
    (_shape(3, 128, 10, 10, 64, 1, 1, seed=242), "2"),
    (_shape(1, 96, 17, 15, 130, 3, 3, pd=(2, 2), dl=(2, 2), seed=243), "7"),
    (_shape(2, 16, 13, 11, 70, 3, 3, pd=(1, 1), seed=244), "3"),
]


# "-io": NHWC x and y, so the tail tiles go out through the NHWC epilogue
@pytest.mark.parametrize("dt", ["f32", "bf16", "bf16-nhwc", "f32-nhwc-io", "bf16-nhwc-io"])
@pytest.mark.parametrize("idx", range(len(TAIL)))
def test_tail_split(idx, dt):
    import torch
    base, force = TAIL[idx]
    f32 = dt.startswith("f32")
    cs = base.with_(x_dtype="f32" if f32 else "bf16", y_dtype="f32" if f32 else "bf16",
                    layout="nhwc" if dt.endswith("-io") else "nchw")
    kernel = "nhwc" if "nhwc" in dt else "0"
    if dt.startswith("bf16-nhwc") and not _nhwc_ok(cs):
        pytest.skip("the NHWC gather needs C/g a multiple of 32")
    if dt == "f32-nhwc-io" and (cs.c // cs.groups) % 16 != 0:
        pytest.skip("the fp32 NHWC gather needs C/g a multiple of 16")
    env = {"CONV2D_TAIL": force, "CONV2D_KSPLIT": "1"}
    old = {k: os.environ.get(k) for k in env}
    os.environ.update(env)
    try:
        for mode, c in (("random", cs), ("integer", cs.with_(y_dtype="f32"))):
            print(f"\n[case] tail {c} kernel={kernel} mode={mode}", flush=True)
            with _Kernel(kernel):
                dc = DeviceConv(c, mode)
            try:
                plan = dc.plan(IMPLICIT)
                assert plan.kernel == B.CONV2D_KERNEL_GEMM and plan.ksplit == 1
                assert plan.tail_tiles > 0 and plan.tail_pieces == int(force), (plan.tail_tiles, plan.tail_pieces)
                assert plan.needs_reorder == (0 if dt.endswith("-io") else plan.needs_reorder)
                ys = []
                for _ in range(2):
                    dc.run(IMPLICIT)
                    torch.cuda.synchronize()
                    ys.append(dc.y_nchw())
                inputs = (dc.x_host, dc.w_host, dc.b_host)
            finally:
                dc.close()
            assert np.array_equal(ys[0], ys[1])
            y_ref, a_ref = _reference(c, mode, inputs)
            if mode == "integer":
                bad = np.argwhere(ys[0] != y_ref)
                assert bad.size == 0, f"{len(bad)} mismatches, first at {bad[0]}"
            else:
                _, pt = oracle.normalised_errors(ys[0], y_ref, a_ref)
                gate = GATE[c.x_dtype] if c.y_dtype == "f32" else max(GATE[c.x_dtype], 2.0 ** -8)
                assert pt <= gate, f"per-point error {pt:.3e} > {gate}"
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def test_tail_split_planned_cfg2_repeat():
    """cfg2 as planned (1568 tiles: 32 in 6 pieces of 3 of its 18 stages) run three times on one
    descriptor, each result identical and on the oracle's sampled outputs."""
    import torch
    cs = datagen.CONFIGS["cfg2"]
    dc = DeviceConv(cs, "random")
    try:
        plan = dc.plan(IMPLICIT)
        assert plan.tail_tiles == 32 and plan.tail_pieces == 6
        ys = []
        for _ in range(3):
            dc.run(IMPLICIT)
            torch.cuda.synchronize()
            ys.append(dc.y_nchw())
        inputs = (dc.x_host, dc.w_host, dc.b_host)
    finally:
        dc.close()
    assert np.array_equal(ys[0], ys[1]) and np.array_equal(ys[0], ys[2])
    y_ref, a_ref = _reference(cs, "random", inputs)
    _, pt = oracle.normalised_errors(ys[0], y_ref, a_ref)
    assert pt <= GATE["f32"]


def test_tail_split_soak_cfg2():
    """cfg2 as planned (its last 32 tiles each summed from 6 pieces that may run on different
    XCDs, handed over through device-scope stores and an arrival counter) called 2000 times back
    to back into a ring of outputs; each result is compared bit for bit with the first on the
    stream itself, and the test stops at the first mismatch."""
    import torch
    cs = datagen.CONFIGS["cfg2"]
    dc = DeviceConv(cs, "random")
    try:
        assert dc.plan(IMPLICIT).tail_tiles > 0
        stream = torch.cuda.current_stream()
        dc.run(IMPLICIT, stream)
        torch.cuda.synchronize()
        ref = dc.y.clone()
        ring = [torch.empty_like(dc.y) for _ in range(8)]
        bad = torch.zeros((), dtype=torch.int64, device=dc.y.device)
        for i in range(2000):
            y = ring[i % 8]
            B.conv2d_fwd(dc.desc, dc.x, dc.w, dc.b, y, IMPLICIT, stream)
            bad += (y != ref).any().to(torch.int64)
            if i % 250 == 249:
                torch.cuda.synchronize()
                assert int(bad) == 0, f"a result differed from the first by call {i}"
        torch.cuda.synchronize()
        assert int(bad) == 0
    finally:
        dc.close()


def test_descriptor_shared_across_streams():
    """One descriptor (cfg2 as planned: tail-split partials and arrival counters and the
    tap-major filter copy in its workspaces) called on two streams in turn without any
    synchronisation between the calls: each call on the other stream waits for the previous
    one, so every result equals the one of a call on the current stream alone."""
    import torch
    cs = datagen.CONFIGS["cfg2"]
    dc = DeviceConv(cs, "random")
    try:
        assert dc.plan(IMPLICIT).tail_tiles > 0
        dc.run(IMPLICIT)
        torch.cuda.synchronize()
        ref = dc.y.clone()
        streams = [torch.cuda.Stream(), torch.cuda.Stream()]
        outs = [torch.empty_like(dc.y) for _ in range(24)]
        torch.cuda.synchronize()
        for i, y in enumerate(outs):
            B.conv2d_fwd(dc.desc, dc.x, dc.w, dc.b, y, IMPLICIT, streams[i % 2])
        torch.cuda.synchronize()
        bad = [i for i, y in enumerate(outs) if not torch.equal(y, ref)]
        assert not bad, f"calls {bad} differ from the single-stream result"
    finally:
        dc.close()


# the sliced kernel's last-round split: more tiles than persistent blocks, the tiles past the
# last whole round computed by 4 or 8 blocks each (wave groups of the tile)
SLICE_TAIL = [
    datagen.ConvShape(n=12, c=3, h=224, w=224, k=64, r=7, s=7, stride=(2, 2), pad=(3, 3), seed=340),   # 588 tiles
    datagen.ConvShape(n=11, c=3, h=224, w=224, k=96, r=7, s=7, stride=(2, 2), pad=(3, 3), seed=341),   # 1078 tiles
]


@pytest.mark.parametrize("dt", [("f32", "f32", "nchw"), ("bf16", "bf16", "nchw"), ("f32", "f32", "nhwc")],
                         ids=lambda d: "-".join(d))
@pytest.mark.parametrize("idx", range(len(SLICE_TAIL)))
def test_slice_last_round_split(idx, dt):
    cs = SLICE_TAIL[idx].with_(x_dtype=dt[0], y_dtype=dt[1], layout=dt[2])
    _check(cs, IMPLICIT, "random", kernel="1", waves="8")
    _check(cs, IMPLICIT, "integer", kernel="1", waves="8")


# the sliced kernel's fp32 slices copied 16 bytes per lane (W % 4 == 0): paddings 0 to 4 (slice
# shift 3, 2, 1, 0), strides 1 and 2, row and column dilation, a line filled up to its last
# word, two channel tiles; W % 4 != 0 keeps the 4-byte copies; each shape also with the
# 4-byte copies forced (CONV2D_SLICE_X1), and with one and two slice buffers (CONV2D_SLICE_DB)
X4 = [
    _shape(2, 3, 32, 32, 16, 7, 7, st=(2, 2), pd=(3, 3), seed=370),
    _shape(1, 5, 20, 24, 40, 3, 3, pd=(1, 1), seed=371),
    _shape(1, 3, 16, 16, 8, 5, 5, pd=(2, 2), seed=372),
    _shape(1, 4, 12, 20, 8, 3, 3, seed=373),
    _shape(1, 3, 12, 16, 8, 5, 5, pd=(2, 4), seed=374),
    _shape(2, 3, 20, 28, 70, 3, 3, st=(1, 2), pd=(2, 1), dl=(2, 1), seed=375),
    _shape(1, 2, 6, 248, 8, 3, 5, pd=(1, 2), seed=376),
    _shape(1, 3, 15, 18, 8, 3, 3, pd=(1, 1), seed=377),
]


@pytest.mark.parametrize("db", ["1", "0"], ids=["two-buffers", "one-buffer"])
@pytest.mark.parametrize("copy", ["x4", "x1"])
@pytest.mark.parametrize("waves", ["4", "8", "16"])
@pytest.mark.parametrize("idx", range(len(X4)))
def test_slice_x4_copies(idx, waves, copy, db):
    cs = X4[idx]
    with _Env(CONV2D_SLICE_X1="1" if copy == "x1" else "", CONV2D_SLICE_DB=db):
        _check(cs, IMPLICIT, kernel="1", waves=waves)
        _check(cs, IMPLICIT, "integer", kernel="1", waves=waves)


# the sliced kernel's packed-row bf16 layout: input pairs per LDS word, filter rows padded to 8
# taps; odd and even padding (slice shift 1 / 0), strides 1 and 2 (window starts of both
# parities), 1 to 8 taps per row, row dilation, rectangular filters, two channel tiles, groups
PACKED = [
    _shape(2, 3, 17, 20, 40, 3, 3, pd=(1, 1), seed=360),
    _shape(1, 5, 16, 30, 70, 5, 5, st=(2, 2), pd=(2, 2), seed=361),
    _shape(2, 2, 21, 24, 16, 7, 7, st=(2, 2), pd=(3, 3), seed=362),
    _shape(1, 4, 12, 14, 33, 8, 8, seed=363),
    _shape(1, 3, 9, 10, 20, 1, 1, seed=364),
    _shape(2, 6, 15, 18, 24, 3, 2, st=(2, 1), pd=(2, 1), dl=(2, 1), seed=365),
    _shape(1, 8, 13, 16, 48, 3, 3, st=(1, 2), pd=(1, 1), g=2, seed=366),
    _shape(3, 1, 40, 46, 96, 7, 5, st=(2, 3), pd=(3, 2), seed=367),
    # wider rows, paddings 2, 0, 3, 7, 8-tap rows
    _shape(1, 3, 20, 32, 24, 5, 5, pd=(2, 2), seed=368),
    _shape(2, 2, 18, 40, 16, 3, 3, seed=369),
    _shape(1, 4, 15, 48, 40, 7, 7, st=(2, 2), pd=(3, 3), seed=402),
    _shape(1, 3, 12, 24, 16, 8, 8, pd=(4, 7), seed=403),
]


@pytest.mark.parametrize("mode", ["random", "integer"])
@pytest.mark.parametrize("ydt", ["bf16", "f32"])
@pytest.mark.parametrize("idx", range(len(PACKED)))
def test_slice_packed_rows(idx, ydt, mode):
    cs = PACKED[idx].with_(x_dtype="bf16", y_dtype=ydt)
    with _Kernel("1", "8"):
        d = B.conv2d_desc_create(params_for(cs))
        try:
            plan = B.conv2d_plan_query(d, IMPLICIT)
        finally:
            B.conv2d_desc_destroy(d)
    rows = (cs.c // cs.groups) * cs.r
    assert plan.kernel == B.CONV2D_KERNEL_SLICE and plan.kred_pad == 16 * ((rows + 1) // 2)
    _check(cs, IMPLICIT, mode, kernel="1", waves="8")


@pytest.mark.parametrize("idx", [2, 1], ids=["elementwise-slice", "gemm"])
def test_slice_packed_rows_unaligned_input(idx):
    """An x that starts 2 bytes past a 4-byte boundary takes the element-wise slice layout (or,
    when only the packed layout fits LDS, the tiled GEMM) and gives a result on the oracle's
    gate, equal to the aligned one when the element-wise slice runs."""
    import torch
    cs = PACKED[idx].with_(x_dtype="bf16", y_dtype="bf16")
    x, w, b = datagen.make_inputs(cs, "random")
    dev = torch.device("cuda:0")
    xb = torch.from_numpy(x).to(dev).to(torch.bfloat16)
    store = torch.empty(x.size + 1, dtype=torch.bfloat16, device=dev)
    xo = store[1:].view(x.shape)
    xo.copy_(xb)
    wb = torch.from_numpy(w).to(dev).to(torch.bfloat16)
    bb = torch.from_numpy(b).to(dev)
    assert xo.data_ptr() % 4 == 2
    outs = []
    with _Kernel("1", "8"):
        for xx in (xb, xo):
            dc = DeviceConv(cs, device_inputs=(xx, wb, bb))
            try:
                dc.run(IMPLICIT)
                torch.cuda.synchronize()
                outs.append(dc.y.clone())
            finally:
                dc.close()
    if idx == 2:
        assert torch.equal(outs[0], outs[1])
    y_ref, a_ref = oracle.conv2d(x, w, b, cs.stride, cs.pad, cs.dil, cs.groups)
    for y in outs:
        _, pt = oracle.normalised_errors(y.float().cpu().numpy().astype(np.float64), y_ref, a_ref)
        assert pt <= 2.0 ** -8


# grouped layers on the direct kernel (C/g > 1 or K/g > 1): per-group output channel chunks
# of 1/2/4/8/16, input channels staged in chunks when the window and filters do not fit at
# once, bands of output rows, strides, dilations, rectangular filters, ragged sizes
GROUPED = [
    _shape(2, 16, 11, 13, 16, 3, 3, pd=(1, 1), g=8, seed=250),            # C/g 2, K/g 2
    _shape(1, 24, 9, 10, 8, 3, 3, pd=(1, 1), g=8, seed=251),              # C/g 3, K/g 1
    _shape(2, 32, 14, 14, 32, 3, 3, pd=(1, 1), g=8, seed=252),            # 4, 4
    _shape(1, 64, 17, 15, 64, 3, 3, st=(2, 2), pd=(1, 1), g=8, seed=253), # 8, 8, strided
    _shape(1, 48, 12, 12, 96, 5, 3, pd=(2, 1), dl=(1, 2), g=3, seed=254), # 16, 32 (two chunks), dilated
    _shape(1, 96, 9, 9, 120, 3, 3, pd=(2, 2), dl=(2, 2), g=3, seed=255),  # 32, 40 (three chunks)
    _shape(1, 128, 10, 9, 48, 7, 7, pd=(3, 3), g=2, seed=256),            # 64 channels in chunks of 2
    _shape(2, 12, 40, 33, 18, 3, 3, st=(1, 2), pd=(1, 1), g=6, seed=257), # 2, 3, bands of rows
    _shape(1, 8, 70, 700, 16, 1, 1, g=4, seed=258),                       # rows too wide: generic kernel
    _shape(1, 6, 5, 5, 12, 5, 5, pd=(2, 2), g=6, seed=259),               # C/g 1, K/g 2 (multiplier)
    _shape(2, 40, 13, 11, 20, 3, 3, pd=(1, 1), g=10, seed=260),           # 4, 2: groups 4 to a block, 2 left
    _shape(1, 24, 31, 29, 72, 3, 3, st=(2, 2), pd=(1, 1), g=12, seed=261),# 2, 6: 8 groups to a block
]


class _Env:
    def __init__(self, **env):
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


# strip = "1": the row-strip kernel where it applies (square filters, strides 1/2, no dilation),
# "0": the per-pixel grouped kernel for every shape
@pytest.mark.parametrize("strip", ["1", "0"], ids=["strip", "perpixel"])
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("idx", range(len(GROUPED)))
def test_grouped_direct(idx, dt, strip):
    cs = GROUPED[idx].with_(x_dtype=dt, y_dtype=dt)
    with _Env(CONV2D_GROUPED_STRIP=strip):
        _check(cs, DIRECT)
        _check(cs.with_(y_dtype="f32"), DIRECT, "integer")


# the row-strip grouped kernel: every filter size and stride it takes, 1 to 8 output channels
# per strip and chunks of 8 beyond, channels staged in chunks, rows that are not a multiple of
# 4 (element-wise staging, ragged last strip), bands of rows, groups batched per block
STRIP = [
    _shape(2, 128, 56, 56, 128, 3, 3, pd=(1, 1), g=32, seed=380),           # C/g 4, K/g 4
    _shape(1, 64, 30, 30, 64, 3, 3, st=(2, 2), pd=(1, 1), g=8, seed=381),   # 8, 8, stride 2
    _shape(2, 24, 17, 19, 48, 5, 5, pd=(2, 2), g=6, seed=382),              # 4, 8, W % 4 != 0
    _shape(1, 32, 28, 28, 96, 1, 1, g=8, seed=383),                         # 4, 12: two chunks of 8
    _shape(1, 6, 40, 41, 9, 7, 7, st=(2, 2), pd=(3, 3), g=3, seed=384),     # 2, 3
    _shape(2, 40, 23, 22, 20, 3, 3, pd=(1, 1), g=20, seed=385),             # 2, 1
    _shape(1, 256, 14, 14, 32, 3, 3, pd=(1, 1), g=2, seed=386),             # 128 channels in chunks
    _shape(3, 16, 9, 300, 16, 3, 3, pd=(1, 1), g=4, seed=387),              # wide rows, one row per band
]


@pytest.mark.parametrize("dt", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")], ids=lambda d: "-".join(d))
@pytest.mark.parametrize("idx", range(len(STRIP)))
def test_grouped_strip(idx, dt):
    cs = STRIP[idx].with_(x_dtype=dt[0], y_dtype=dt[1])
    _check(cs, DIRECT)
    if dt[1] == "f32":
        _check(cs, DIRECT, "integer")


# the streamed-row depthwise kernel (stride 1; 3x3 at dilation 1 or 2, 5x5 and 7x7 at
# dilation 1): bands of rows (ragged last band and strip), odd and even padding (bf16 words
# start at the strip or one value before it), multiplier 2, asymmetric and zero padding, no
# bias, wide rows with one unit per wave, first and last input planes (word-by-word loads);
# shapes it does not take (odd W in bf16, 7x7 at dilation 2) go to the block-per-plane
# kernel, through which every shape also runs with rows = "0"
DW_ROWS = [
    _shape(2, 16, 56, 56, 16, 3, 3, pd=(1, 1), g=16, seed=390),             # 4 bands of 14
    _shape(1, 8, 37, 37, 8, 5, 5, pd=(2, 2), g=8, seed=391),                # Wo % 4 != 0, 32 KiB
    _shape(2, 6, 30, 30, 12, 3, 3, pd=(1, 1), g=6, seed=392),               # multiplier 2
    _shape(1, 4, 33, 64, 4, 7, 7, pd=(3, 3), g=4, seed=393),                # two copies per row
    _shape(1, 4, 50, 60, 4, 3, 3, pd=(2, 2), dl=(2, 2), g=4, seed=394),     # dilation 2
    _shape(1, 3, 45, 40, 3, 7, 7, pd=(6, 6), dl=(2, 2), g=3, seed=395),     # not taken (7x7 d2)
    _shape(1, 2, 20, 250, 2, 3, 3, pd=(1, 1), g=2, seed=396),               # one unit per wave
    _shape(2, 5, 29, 27, 5, 3, 3, g=5, seed=397, bias=False),               # no padding, no bias
    _shape(1, 4, 21, 32, 4, 5, 5, pd=(1, 3), g=4, seed=398),                # ph != pw, Wo = 34
    _shape(3, 8, 14, 14, 8, 3, 3, pd=(1, 1), g=8, seed=399),                # 16 units per wave
    _shape(2, 4, 23, 31, 4, 3, 3, pd=(1, 1), g=4, seed=400),                # odd W (bf16: not taken)
    _shape(1, 2, 26, 70, 2, 5, 5, pd=(2, 2), g=2, seed=401),                # 2 planes: all edge waves
]


@pytest.mark.parametrize("rows", ["1", "0"], ids=["rows", "block"])
@pytest.mark.parametrize("dt", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")], ids=lambda d: "-".join(d))
@pytest.mark.parametrize("idx", range(len(DW_ROWS)))
def test_depthwise_rows(idx, dt, rows):
    cs = DW_ROWS[idx].with_(x_dtype=dt[0], y_dtype=dt[1])
    with _Env(CONV2D_DW_ROWS=rows):
        _check(cs, DIRECT)
        if dt[1] == "f32":
            _check(cs, DIRECT, "integer")


# the streamed-row kernel's block size: one wave per block or 4 independent waves (the plan takes
# 4 for 3x3 planes up to 32 columns); forced both ways on every 3x3 dilation-1 shape, so the
# last block's waves past the final unit are covered at several unit counts
@pytest.mark.parametrize("wpb", ["1", "4"])
@pytest.mark.parametrize("dt", [("f32", "f32"), ("bf16", "bf16")], ids=lambda d: "-".join(d))
@pytest.mark.parametrize("idx", [i for i, c in enumerate(DW_ROWS) if c.r == 3 and c.dil == (1, 1)])
def test_depthwise_rows_block_size(idx, dt, wpb):
    cs = DW_ROWS[idx].with_(x_dtype=dt[0], y_dtype=dt[1])
    with _Env(CONV2D_DW_ROWS="1", CONV2D_DWR_WPB=wpb):
        _check(cs, DIRECT)


# NHWC <-> NCHW copies: the 64x64 vector kernel (both sides multiples of 4, ragged tiles) and the
# 32x32 element kernel (CONV2D_TRANSPOSE32, and sides that are not multiples of 4), through NHWC
# convolutions that reorder x and y
TRANSPOSE = [
    _shape(2, 64, 14, 14, 64, 3, 3, pd=(1, 1), seed=410),
    _shape(1, 36, 9, 20, 12, 3, 3, seed=411),
    _shape(1, 12, 7, 9, 16, 1, 1, seed=412),
    _shape(2, 200, 10, 10, 24, 3, 3, pd=(1, 1), seed=413),
]


@pytest.mark.parametrize("kernel", ["64", "32"])
@pytest.mark.parametrize("dt", [("f32", "f32"), ("bf16", "bf16")], ids=lambda d: d[0])
@pytest.mark.parametrize("idx", range(len(TRANSPOSE)))
def test_layout_transposes(idx, dt, kernel):
    cs = TRANSPOSE[idx].with_(layout="nhwc", x_dtype=dt[0], y_dtype=dt[1])
    with _Env(CONV2D_TRANSPOSE32="1" if kernel == "32" else ""):
        for algo in (IMPLICIT, IM2COL):
            _check(cs, algo)
            if dt[1] == "f32":
                _check(cs, algo, "integer")


# Winograd F(2x2, 3x3): 3x3, stride 1, dilation 1, one group, fp32; odd output sizes (clipped
# 2x2 tiles), paddings 0/1/2, channel counts across GEMM tiles, NHWC, chunked tiles
WINOGRAD = B.CONV2D_ALGO_WINOGRAD
WINO = [
    _shape(1, 3, 9, 11, 5, 3, 3, pd=(1, 1), seed=270),
    _shape(2, 17, 13, 10, 33, 3, 3, seed=271),
    _shape(1, 70, 15, 15, 90, 3, 3, pd=(2, 2), seed=272),
    _shape(3, 64, 14, 14, 128, 3, 3, pd=(1, 1), seed=273),
    _shape(2, 24, 8, 31, 16, 3, 3, pd=(1, 0), seed=274, bias=False),
    # W a multiple of 4 with padding 1 or 0: the F(4x4) input transform's 16-byte row loads
    _shape(2, 20, 13, 16, 24, 3, 3, pd=(1, 1), seed=275),
    _shape(1, 33, 9, 20, 17, 3, 3, seed=276),
]


# F(2x2): the transforms hold integers and halves, so integer data stays exact; F(4x4): the
# filter transform has sixths and 24ths, so integer data is checked against the gate
@pytest.mark.parametrize("mt", [2, 4])
@pytest.mark.parametrize("idx", range(len(WINO)))
def test_winograd(idx, mt, monkeypatch):
    monkeypatch.setenv("CONV2D_WINO_TILE", str(mt))
    cs = WINO[idx]
    dc = DeviceConv(cs, "random")
    try:
        assert dc.plan(WINOGRAD).wino_tile == mt
    finally:
        dc.close()
    _check(cs, WINOGRAD)
    _check(cs, WINOGRAD, "integer", exact=mt == 2)
    _check(cs.with_(layout="nhwc"), WINOGRAD)


# bf16 Winograd (F(2x2), C a multiple of 8): U and V rounded to bf16, fp32 GEMM sums; NCHW and
# NHWC inputs, bf16 and fp32 outputs, chunked tiles; integer data stays exact (the transforms
# only add, subtract and halve small integers)
WINO_BF16 = [
    _shape(3, 64, 14, 14, 128, 3, 3, pd=(1, 1), seed=277),
    _shape(2, 24, 8, 31, 16, 3, 3, pd=(1, 0), seed=278, bias=False),
    _shape(1, 128, 9, 13, 72, 3, 3, pd=(1, 1), seed=279),
    _shape(2, 16, 12, 12, 40, 3, 3, seed=280),
]


@pytest.mark.parametrize("var", [("nchw", "bf16"), ("nhwc", "bf16"), ("nchw", "f32")], ids=lambda v: "-".join(v))
@pytest.mark.parametrize("idx", range(len(WINO_BF16)))
def test_winograd_bf16(idx, var):
    layout, ydt = var
    cs = WINO_BF16[idx].with_(layout=layout, x_dtype="bf16", y_dtype=ydt)
    dc = DeviceConv(cs, "random")
    try:
        p = dc.plan(WINOGRAD)
        assert p.wino_tile == 2 and p.needs_reorder == 1
    finally:
        dc.close()
    _check(cs, WINOGRAD)
    _check(cs.with_(y_dtype="f32"), WINOGRAD, "integer")


def test_winograd_bf16_chunks(monkeypatch):
    cs = WINO_BF16[0].with_(x_dtype="bf16", y_dtype="bf16")
    monkeypatch.setenv("CONV2D_WORKSPACE_LIMIT_BYTES", str(16 * (64 * 2 + 128 * 4) * 40))
    dc = DeviceConv(cs, "random")
    try:
        assert dc.plan(WINOGRAD).chunks > 1
    finally:
        dc.close()
    _check(cs, WINOGRAD)
    _check(cs.with_(y_dtype="f32"), WINOGRAD, "integer")


@pytest.mark.parametrize("mt", [2, 4])
def test_winograd_chunks_and_configs(mt, monkeypatch):
    # a workspace cap that forces several chunks of tiles
    monkeypatch.setenv("CONV2D_WINO_TILE", str(mt))
    cs = WINO[3]
    npos = (mt + 2) ** 2
    monkeypatch.setenv("CONV2D_WORKSPACE_LIMIT_BYTES", str(npos * (64 + 128) * 4 * 40))
    dc = DeviceConv(cs, "random")
    try:
        assert dc.plan(WINOGRAD).chunks > 1
    finally:
        dc.close()
    _check(cs, WINOGRAD)
    _check(cs, WINOGRAD, "integer", exact=mt == 2)
    monkeypatch.delenv("CONV2D_WORKSPACE_LIMIT_BYTES")
    _check(datagen.CONFIGS["cfg2"], WINOGRAD)


# 32-row tiles (layers with few output channels per group): forced on ragged and tiny K,
# grouped layers, through every gather (NCHW table and tap-major, bf16 NHWC) and the explicit
# path's dense GEMM, fp32 (BK 16, both prefetch distances) and bf16
SMALL_M = [
    _shape(2, 32, 15, 13, 3, 3, 3, pd=(1, 1), seed=290),
    _shape(1, 64, 20, 18, 16, 5, 5, pd=(2, 2), seed=291),
    _shape(2, 48, 11, 23, 33, 3, 3, st=(2, 1), pd=(1, 1), seed=292),
    _shape(1, 64, 14, 14, 48, 3, 3, pd=(2, 2), dl=(2, 2), g=2, seed=293),
    _shape(3, 16, 9, 9, 20, 1, 1, seed=294),
]


@pytest.mark.parametrize("algo", [IMPLICIT, IM2COL], ids=lambda a: ALGO_IDS[a])
@pytest.mark.parametrize("dt", ["f32", "f32-pf2", "bf16", "bf16-nhwc"])
@pytest.mark.parametrize("tile", [5, 6], ids=["32x128", "32x256"])
@pytest.mark.parametrize("idx", range(len(SMALL_M)))
def test_small_m_tiles(idx, tile, dt, algo, monkeypatch):
    cs = SMALL_M[idx].with_(x_dtype="f32" if dt.startswith("f32") else "bf16",
                            y_dtype="f32" if dt.startswith("f32") else "bf16")
    monkeypatch.setenv("CONV2D_GEMM", f"k32:{tile}:16:2" if dt == "f32-pf2" else f"k32:{tile}")
    kernel = "nhwc" if dt == "bf16-nhwc" else "0"
    if algo == IM2COL and dt == "bf16-nhwc":
        pytest.skip("the NHWC gather is an implicit-path source")
    with _Kernel(kernel):
        dc = DeviceConv(cs, "random")
    try:
        p = dc.plan(algo)
        assert (p.tile_m, p.tile_n) == (32, 128 if tile == 5 else 256), (p.tile_m, p.tile_n)
    finally:
        dc.close()
    _check(cs, algo, "random", kernel)
    _check(cs.with_(y_dtype="f32"), algo, "integer", kernel)


# few output channels (ungrouped, K <= 4) on the vector-ALU direct kernel: every K and filter
# size, strides, dilations, paddings, ragged pixel blocks, one channel, channel ranges forced to
# 1 / 3 / 7 (partials added by the unpack kernel) and the planner's count
SMALLK = [
    _shape(2, 40, 17, 15, 3, 3, 3, pd=(1, 1), seed=300),
    _shape(1, 9, 23, 21, 1, 7, 7, st=(2, 2), pd=(3, 3), seed=301),
    _shape(3, 33, 12, 14, 4, 5, 5, pd=(4, 4), dl=(2, 2), seed=302),
    _shape(2, 64, 9, 11, 2, 1, 1, seed=303, bias=False),
    _shape(1, 1, 10, 10, 3, 3, 3, st=(1, 2), pd=(0, 1), seed=304),
]


# NHWC x and y through the NHWC gather: the GEMM's epilogue writes NHWC y itself (four adjacent
# channels per 16-byte fp32 or 8-byte bf16 store when K/g is a multiple of 4, one element per
# store otherwise), so neither x nor y is reordered.  Groups, bias, ragged
# pixel and channel tiles, K/g = 30 and 33, strides, padding and dilation.
NHWC_EPI = [
    _shape(2, 64, 15, 17, 96, 3, 3, pd=(1, 1), seed=230),
    _shape(1, 128, 14, 14, 64, 3, 3, pd=(1, 1), g=2, seed=231),
    _shape(3, 32, 11, 9, 30, 3, 3, st=(2, 2), pd=(1, 1), seed=232),
    _shape(2, 64, 12, 12, 66, 1, 1, g=2, seed=233),
    _shape(1, 32, 9, 13, 40, 5, 5, pd=(4, 4), dl=(2, 2), seed=234, bias=False),
    _shape(2, 96, 7, 7, 200, 3, 3, pd=(1, 1), seed=235),
]


@pytest.mark.parametrize("dt", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")], ids=lambda d: "-".join(d))
@pytest.mark.parametrize("idx", range(len(NHWC_EPI)))
def test_nhwc_epilogue(idx, dt):
    import torch
    cs = NHWC_EPI[idx].with_(layout="nhwc", x_dtype=dt[0], y_dtype=dt[1])
    with _Kernel("nhwc"):
        dc = DeviceConv(cs, "random", timing=B.CONV2D_TIMING_PHASES)
    try:
        p = dc.plan(IMPLICIT)
        assert p.kernel == B.CONV2D_KERNEL_GEMM
        assert p.needs_reorder == 0
        dc.run(IMPLICIT)
        torch.cuda.synchronize()
        calls = dc.breakdown(IMPLICIT)["calls"]
        # pre-convolution reordering: only the filters' tap-major repack (R*S > 1), never x
        assert calls["pre_reorder"] == (1 if cs.r * cs.s > 1 else 0), calls
        assert calls["post_reorder"] == 0, calls
    finally:
        dc.close()
    _check(cs, IMPLICIT, "random", "nhwc")
    _check(cs.with_(y_dtype="f32"), IMPLICIT, "integer", "nhwc")


# the sliced kernel with NHWC x and y: x is reordered to NCHW first, y written NHWC by the
# kernel (4 adjacent channels per store when K/g is a multiple of 4, element stores otherwise),
# so no post-convolution reorder; 7x7 stride-2 stem (Wo = 125), K/g = 30, groups, two channel tiles
SLICE_NHWC = [
    _shape(1, 3, 22, 250, 64, 7, 7, st=(2, 2), pd=(3, 3), seed=250),
    _shape(1, 3, 30, 30, 30, 3, 3, pd=(1, 1), seed=251),
    _shape(2, 8, 20, 21, 48, 3, 3, pd=(1, 1), g=2, seed=252),
    _shape(1, 4, 17, 19, 100, 3, 3, pd=(1, 1), seed=253, bias=False),
]


@pytest.mark.parametrize("dt", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")], ids=lambda d: "-".join(d))
@pytest.mark.parametrize("idx", range(len(SLICE_NHWC)))
def test_slice_nhwc_output(idx, dt):
    import torch
    cs = SLICE_NHWC[idx].with_(layout="nhwc", x_dtype=dt[0], y_dtype=dt[1])
    with _Kernel("1"):
        dc = DeviceConv(cs, "random", timing=B.CONV2D_TIMING_PHASES)
    try:
        assert dc.plan(IMPLICIT).kernel == B.CONV2D_KERNEL_SLICE
        dc.run(IMPLICIT)
        torch.cuda.synchronize()
        calls = dc.breakdown(IMPLICIT)["calls"]
        assert calls["pre_reorder"] == 1 and calls["post_reorder"] == 0, calls
    finally:
        dc.close()
    _check(cs, IMPLICIT, "random", "1")
    _check(cs.with_(y_dtype="f32"), IMPLICIT, "integer", "1")


# depthwise layers with NHWC x and y on the NHWC depthwise kernel (4 channels x 4 or 8 output
# pixels per thread, filters reordered to [R*S][C]): 3x3, 5x5 at stride 2, dilation 2, 1x1,
# rectangular, ragged rows (Wo not a multiple of 4 or 8), C = 4 and 12, no bias
DW_NHWC = [
    _shape(2, 64, 15, 17, 64, 3, 3, pd=(1, 1), g=64, seed=260),
    _shape(1, 32, 23, 21, 32, 5, 5, st=(2, 2), pd=(2, 2), g=32, seed=261),
    _shape(2, 12, 13, 14, 12, 3, 3, pd=(2, 2), dl=(2, 2), g=12, seed=262, bias=False),
    _shape(3, 4, 9, 10, 4, 1, 1, g=4, seed=263),
    _shape(1, 128, 7, 9, 128, 3, 5, st=(1, 2), pd=(1, 2), g=128, seed=264),
    # stride 1, dilation 1, S <= 7: 8 pixels per thread, shared input columns loaded once per
    # row; 7x7, 5x3 with Wo = 17, and S = 9 (beyond the shared-column path)
    _shape(1, 16, 11, 13, 16, 7, 7, pd=(3, 3), g=16, seed=265),
    _shape(2, 8, 6, 19, 8, 5, 3, pd=(2, 0), g=8, seed=266),
    _shape(1, 4, 5, 20, 4, 1, 9, pd=(0, 4), g=4, seed=267),
]


@pytest.mark.parametrize("dt", [("f32", "f32"), ("bf16", "bf16"), ("bf16", "f32")], ids=lambda d: "-".join(d))
@pytest.mark.parametrize("idx", range(len(DW_NHWC)))
def test_depthwise_nhwc(idx, dt):
    import torch
    cs = DW_NHWC[idx].with_(layout="nhwc", x_dtype=dt[0], y_dtype=dt[1])
    dc = DeviceConv(cs, "random", timing=B.CONV2D_TIMING_PHASES)
    try:
        assert dc.plan(DIRECT).needs_reorder == 0
        dc.run(DIRECT)
        torch.cuda.synchronize()
        calls = dc.breakdown(DIRECT)["calls"]
        # pre-convolution reordering: the filters only
        assert calls["pre_reorder"] == 1 and calls["post_reorder"] == 0, calls
    finally:
        dc.close()
    _check(cs, DIRECT, "random")
    _check(cs.with_(y_dtype="f32"), DIRECT, "integer")


# split reductions with NHWC x and y: the unpack adds the partials and writes NHWC y (16- or
# 8-byte stores of 4 channels when K/g is a multiple of 4), forced to 2, 3 and 5 splits
@pytest.mark.parametrize("ksplit", ["2", "3", "5"])
@pytest.mark.parametrize("dt", [("f32", "f32"), ("bf16", "bf16")], ids=lambda d: "-".join(d))
@pytest.mark.parametrize("idx", range(len(NHWC_EPI)))
def test_nhwc_split_unpack(idx, dt, ksplit, monkeypatch):
    import torch
    cs = NHWC_EPI[idx].with_(layout="nhwc", x_dtype=dt[0], y_dtype=dt[1])
    monkeypatch.setenv("CONV2D_KSPLIT", ksplit)
    monkeypatch.setenv("CONV2D_TAIL", "0")
    with _Kernel("nhwc"):
        dc = DeviceConv(cs, "random", timing=B.CONV2D_TIMING_PHASES)
    try:
        p = dc.plan(IMPLICIT)
        assert p.kernel == B.CONV2D_KERNEL_GEMM and p.needs_reorder == 0
        if p.ksplit <= 1:
            pytest.skip("reduction too short for the forced split")
        dc.run(IMPLICIT)
        torch.cuda.synchronize()
        calls = dc.breakdown(IMPLICIT)["calls"]
        assert calls["in_unpacking"] == 1 and calls["post_reorder"] == 0, calls
    finally:
        dc.close()
    _check(cs, IMPLICIT, "random", "nhwc")
    _check(cs.with_(y_dtype="f32"), IMPLICIT, "integer", "nhwc")


@pytest.mark.parametrize("ranges", [None, "1", "3", "7"])
@pytest.mark.parametrize("var", [("nchw", "f32", "f32"), ("nchw", "bf16", "bf16"), ("nhwc", "bf16", "f32"),
                                 ("nhwc", "f32", "f32")], ids=lambda v: "-".join(v))
@pytest.mark.parametrize("idx", range(len(SMALLK)))
def test_smallk_direct(idx, var, ranges, monkeypatch):
    layout, xdt, ydt = var
    cs = SMALLK[idx].with_(layout=layout, x_dtype=xdt, y_dtype=ydt)
    monkeypatch.setenv("CONV2D_SMALLK", "1")
    if ranges is not None:
        monkeypatch.setenv("CONV2D_SMALLK_RANGES", ranges)
    dc = DeviceConv(cs, "random")
    try:
        p = dc.plan(DIRECT)
        assert p.kernel == B.CONV2D_KERNEL_DIRECT and p.workspace_bytes == (p.ksplit * cs.k * 4 * dc.out_nkhw[0] *
                                                                            dc.out_nkhw[2] * dc.out_nkhw[3]
                                                                            if p.ksplit > 1 else 0)
        if ranges is not None:
            assert max(p.ksplit, 1) == min(int(ranges), cs.c), (p.ksplit, ranges)
    finally:
        dc.close()
    _check(cs, DIRECT, "random")
    _check(cs.with_(y_dtype="f32"), DIRECT, "integer")


EDGE_ALGOS = [("implicit", IMPLICIT, None, None), ("implicit-gemm", IMPLICIT, "0", None),
              ("implicit-slice4", IMPLICIT, "1", "4"), ("implicit-slice8", IMPLICIT, "1", "8"),
              ("implicit-nhwc", IMPLICIT, "nhwc", None),
              ("im2col", IM2COL, None, None), ("direct", DIRECT, None, None)]


@pytest.mark.parametrize("algo", EDGE_ALGOS, ids=lambda a: a[0])
@pytest.mark.parametrize("var", VARIANTS, ids=lambda v: "-".join(v))
@pytest.mark.parametrize("idx", range(len(EDGE)))
def test_edge_grid(idx, var, algo):
    layout, xdt, ydt = var
    _, algo, kernel, waves = algo
    cs = EDGE[idx].with_(layout=layout, x_dtype=xdt, y_dtype=ydt)
    _check(cs, algo, "random", kernel, waves)
    _check(cs.with_(y_dtype="f32"), algo, "integer", kernel, waves)


# ------------------------------------------------------------------ behaviour

@pytest.mark.parametrize("algo", [IMPLICIT, IM2COL, DIRECT], ids=lambda a: ALGO_IDS[a])
def test_run_to_run_bitwise_determinism(algo):
    import torch
    cs = _shape(2, 24, 15, 15, 40, 3, 3, pd=(1, 1), seed=7)
    dc = DeviceConv(cs)
    try:
        dc.run(algo)
        torch.cuda.synchronize()
        y1 = dc.y.clone()
        for _ in range(3):
            dc.run(algo)
        torch.cuda.synchronize()
        assert torch.equal(y1, dc.y)
    finally:
        dc.close()


def test_families_agree_with_each_other():
    import torch
    cs = datagen.CONFIGS["cfg2"].with_(n=4)
    dc = DeviceConv(cs)
    try:
        dc.run(IMPLICIT)
        torch.cuda.synchronize()
        y_imp = dc.y_nchw()
        dc.run(IM2COL)
        torch.cuda.synchronize()
        y_exp = dc.y_nchw()
    finally:
        dc.close()
    _, a_ref = oracle.conv2d(dc.x_host, dc.w_host, dc.b_host, cs.stride, cs.pad, cs.dil, cs.groups)
    _, pt = oracle.normalised_errors(y_imp, y_exp, a_ref)
    assert pt <= 2e-5


def test_chunked_explicit_path(monkeypatch):
    monkeypatch.setenv("CONV2D_WORKSPACE_LIMIT_BYTES", "200000")
    cs = _shape(3, 16, 33, 31, 24, 3, 3, st=(1, 2), pd=(1, 1), seed=9)
    import torch
    dc = DeviceConv(cs, timing=B.CONV2D_TIMING_PHASES)
    try:
        assert dc.plan(IM2COL).chunks > 2
        dc.run(IM2COL)
        torch.cuda.synchronize()
        y = dc.y_nchw()
        bd = dc.breakdown(IM2COL)
        assert bd["calls"]["in_packing"] == dc.plan(IM2COL).chunks
    finally:
        dc.close()
    y_ref, a_ref = oracle.conv2d(dc.x_host, dc.w_host, dc.b_host, cs.stride, cs.pad, cs.dil, cs.groups)
    assert oracle.normalised_errors(y, y_ref, a_ref)[1] <= 1e-5


def test_breakdown_phases_and_invariants():
    import torch
    cs = datagen.CONFIGS["cfg1"].with_(layout="nhwc")
    dc = DeviceConv(cs, timing=B.CONV2D_TIMING_PHASES)
    try:
        for algo in (IMPLICIT, IM2COL, DIRECT):
            for _ in range(3):
                dc.run(algo)
        torch.cuda.synchronize()
        for algo in (IMPLICIT, IM2COL, DIRECT):
            bd = dc.breakdown(algo)
            ms, calls = bd["ms"], bd["calls"]
            assert bd["fwd_calls"] == 3 and calls["pre_analysis"] == 1
            assert calls["in_microkernel"] == 3
            # the sliced kernel (cfg1's implicit path) writes NHWC y itself
            post = 0 if dc.plan(algo).kernel == B.CONV2D_KERNEL_SLICE else 3
            assert calls["pre_reorder"] == 3 and calls["post_reorder"] == post
            assert all(v >= 0 for v in ms.values())
            assert bd["operation_ms"] == pytest.approx(sum(ms.values()))
            assert bd["convolution_ms"] == pytest.approx(
                ms["in_tiling"] + ms["in_packing"] + ms["in_microkernel"] + ms["in_unpacking"])
            if algo == IM2COL:
                assert calls["in_packing"] == 3 and calls["in_unpacking"] == 3
                assert bd["pack_is_preconv"] == 1
            else:
                assert "in_packing" in bd["fused"]
        assert dc.breakdown(B.CONV2D_ALGO_AUTO)["algo"] == "direct"
        B.conv2d_breakdown_reset(dc.desc)
        with pytest.raises(B.Conv2dError):
            dc.breakdown(IMPLICIT)
        B.conv2d_set_timing(dc.desc, B.CONV2D_TIMING_TOTAL)
        dc.run(IMPLICIT)
        torch.cuda.synchronize()
        bd = dc.breakdown(IMPLICIT)
        assert bd["total_calls"] == 1 and bd["calls"]["in_microkernel"] == 0
    finally:
        dc.close()


def test_shared_hip_runtime_with_torch():
    import torch
    v = B.conv2d_runtime_version()
    major, minor = (int(t) for t in torch.version.hip.split(".")[:2])
    assert v // 10000000 == major and (v // 100000) % 100 == minor
