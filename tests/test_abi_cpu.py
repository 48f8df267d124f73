"""The C ABI on the CPU: the library loads, exports what the header declares,
and its host-only planning and validation behave (no GPU needed)."""
import os
import re
import subprocess

import pytest

import datagen
import oracle
import paper_2407_10730_amd as cv
from paper_2407_10730_amd import binding as B
from paper_2407_10730_amd.runner import params_for

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "conv2d.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\**(conv2d_\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_function():
    decl = _declared_functions()
    assert set(decl) == set(B.EXPORTS), decl
    lib = cv.load()
    for name in decl:
        assert hasattr(lib, name)
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (conv2d_\w+)", out))
    assert set(decl) <= exported


def _params(**kw):
    base = dict(n=2, c=4, h=9, w=9, k=6, r=3, s=3, stride_h=1, stride_w=1, pad_h=1, pad_w=1,
                dil_h=1, dil_w=1, groups=1, layout=0, x_dtype=0, y_dtype=0, has_bias=1)
    base.update(kw)
    return B.conv2d_params(**base)


@pytest.mark.parametrize("kw,code", [
    (dict(n=0), B.CONV2D_E_INVALID), (dict(k=-1), B.CONV2D_E_INVALID),
    (dict(stride_h=0), B.CONV2D_E_INVALID), (dict(dil_w=0), B.CONV2D_E_INVALID),
    (dict(pad_h=-1), B.CONV2D_E_INVALID), (dict(groups=0), B.CONV2D_E_INVALID),
    (dict(groups=3), B.CONV2D_E_INVALID), (dict(layout=2), B.CONV2D_E_INVALID),
    (dict(x_dtype=5), B.CONV2D_E_INVALID),
    (dict(x_dtype=0, y_dtype=1), B.CONV2D_E_UNSUPPORTED),
    (dict(h=2, pad_h=0), B.CONV2D_E_SHAPE), (dict(w=3, s=2, dil_w=3, pad_w=0), B.CONV2D_E_SHAPE),
])
def test_create_rejects(kw, code):
    with pytest.raises(B.Conv2dError) as ei:
        B.conv2d_desc_create(_params(**kw))
    assert ei.value.status == code


def test_null_pointers_rejected():
    lib = cv.load()
    assert lib.conv2d_desc_create(None, None) == B.CONV2D_E_NULL
    d = B.conv2d_desc_create(_params())
    try:
        assert lib.conv2d_fwd(d, None, None, None, None, 0, None) == B.CONV2D_E_NULL
        assert lib.conv2d_fwd(d, 1, 1, None, 1, 0, None) == B.CONV2D_E_NULL  # bias missing
        assert lib.conv2d_fwd(d, 1, 1, 1, 1, 9, None) == B.CONV2D_E_INVALID
        # the no-allocation entry point checks its arguments the same way, before any HIP call
        assert lib.conv2d_fwd_noalloc(d, None, None, None, None, 0, None) == B.CONV2D_E_NULL
        assert lib.conv2d_fwd_noalloc(d, 1, 1, None, 1, 0, None) == B.CONV2D_E_NULL
        assert lib.conv2d_fwd_noalloc(d, 1, 1, 1, 1, 9, None) == B.CONV2D_E_INVALID
        assert lib.conv2d_fwd_noalloc(None, 1, 1, 1, 1, 0, None) == B.CONV2D_E_NULL
    finally:
        B.conv2d_desc_destroy(d)
    assert lib.conv2d_desc_destroy(None) == 0


def test_output_shape_matches_oracle_over_a_grid():
    checked = 0
    for h in (1, 2, 5, 8, 13):
        for r in (1, 2, 3, 5):
            for st in (1, 2, 3):
                for pd in (0, 1, 3):
                    for dl in (1, 2):
                        kw = dict(h=h, w=h + 1, r=r, s=max(1, r - 1), stride_h=st, stride_w=st,
                                  pad_h=pd, pad_w=pd, dil_h=dl, dil_w=dl)
                        try:
                            ref = oracle.output_dims((2, 4, h, h + 1), (6, 4, r, max(1, r - 1)),
                                                     (st, st), (pd, pd), (dl, dl))
                        except oracle.OracleError:
                            with pytest.raises(B.Conv2dError):
                                B.conv2d_desc_create(_params(**kw))
                            continue
                        d = B.conv2d_desc_create(_params(**kw))
                        assert B.conv2d_output_shape(d) == (2, 6) + ref
                        B.conv2d_desc_destroy(d)
                        checked += 1
    assert checked > 200


def test_breakdown_before_any_call():
    d = B.conv2d_desc_create(_params())
    try:
        with pytest.raises(B.Conv2dError) as ei:
            B.conv2d_breakdown(d, B.CONV2D_ALGO_IMPLICIT_GEMM)
        assert ei.value.status == B.CONV2D_E_NO_DATA
        with pytest.raises(B.Conv2dError) as ei:
            B.conv2d_breakdown(d, B.CONV2D_ALGO_AUTO)
        assert ei.value.status == B.CONV2D_E_NO_DATA
        B.conv2d_set_timing(d, B.CONV2D_TIMING_TOTAL)
        with pytest.raises(B.Conv2dError):
            B.conv2d_set_timing(d, 7)
        B.conv2d_breakdown_reset(d)
    finally:
        B.conv2d_desc_destroy(d)


def test_auto_algorithm_choice_and_classes():
    dw = datagen.CONFIGS["dw"]
    d = B.conv2d_desc_create(params_for(dw))
    info = B.conv2d_plan_query(d)
    assert info.algo == B.CONV2D_ALGO_DIRECT and info.op_class & 4 and info.op_class & 2
    B.conv2d_desc_destroy(d)
    d = B.conv2d_desc_create(params_for(datagen.CONFIGS["cfg2"]))
    info = B.conv2d_plan_query(d)
    assert info.algo == B.CONV2D_ALGO_IMPLICIT_GEMM and info.kred == 576 and info.op_class == 0
    B.conv2d_desc_destroy(d)
    d = B.conv2d_desc_create(params_for(datagen.CONFIGS["cfg3b"]))
    assert B.conv2d_plan_query(d).op_class == 1 | 32
    B.conv2d_desc_destroy(d)


def test_implicit_microkernel_choice(monkeypatch):
    """Short reductions with C/g off the 16-channel stage grid take the sliced kernel; the
    rest the tiled GEMM; CONV2D_SLICE forces either where the slice fits in LDS."""
    def kernel(cs):
        d = B.conv2d_desc_create(params_for(cs))
        try:
            info = B.conv2d_plan_query(d, B.CONV2D_ALGO_IMPLICIT_GEMM)
            return info.kernel, info.kred_pad
        finally:
            B.conv2d_desc_destroy(d)
    monkeypatch.delenv("CONV2D_SLICE", raising=False)
    assert kernel(datagen.CONFIGS["cfg4"]) == (B.CONV2D_KERNEL_SLICE, 152)       # 147 -> 2 x 76
    # bf16 packed rows: 3 x 7 filter rows padded to 8 taps, 22 rows (two per MFMA step) = 176
    assert kernel(datagen.CONFIGS["cfg4_bf16"]) == (B.CONV2D_KERNEL_SLICE, 176)
    monkeypatch.setenv("CONV2D_SLICE_UNPACKED", "1")
    assert kernel(datagen.CONFIGS["cfg4_bf16"]) == (B.CONV2D_KERNEL_SLICE, 160)  # 147 -> 2 x 80
    assert kernel(datagen.CONFIGS["cfg4_bf16"].with_(w=223))[1] == 160          # odd W: element-wise
    monkeypatch.delenv("CONV2D_SLICE_UNPACKED")
    assert kernel(datagen.CONFIGS["cfg4_bf16"].with_(w=223))[1] == 160
    assert kernel(datagen.CONFIGS["cfg4_bf16"].with_(dil=(1, 2)))[1] == 160      # column dilation
    assert kernel(datagen.CONFIGS["cfg1"])[0] == B.CONV2D_KERNEL_SLICE
    assert kernel(datagen.CONFIGS["cfg2"])[0] == B.CONV2D_KERNEL_GEMM
    big = datagen.CONFIGS["cfg4"].with_(c=48)                                    # 2352-long reduction
    assert kernel(big)[0] == B.CONV2D_KERNEL_GEMM
    c16 = datagen.CONFIGS["cfg2"].with_(c=16, h=130, w=130, r=1, s=1, pad=(0, 0))  # tap-major GEMM
    assert kernel(c16)[0] == B.CONV2D_KERNEL_GEMM
    monkeypatch.setenv("CONV2D_SLICE", "0")
    assert kernel(datagen.CONFIGS["cfg4"])[0] == B.CONV2D_KERNEL_GEMM
    monkeypatch.setenv("CONV2D_SLICE", "1")
    assert kernel(c16)[0] == B.CONV2D_KERNEL_SLICE
    assert kernel(datagen.CONFIGS["cfg2"])[0] == B.CONV2D_KERNEL_GEMM           # 64 x 576 filters overflow LDS
    assert kernel(datagen.CONFIGS["cfg2"].with_(c=16))[0] == B.CONV2D_KERNEL_GEMM  # 96 slice lines
    assert kernel(big)[0] == B.CONV2D_KERNEL_GEMM
    d = B.conv2d_desc_create(params_for(datagen.CONFIGS["dw"]))
    assert B.conv2d_plan_query(d).kernel == B.CONV2D_KERNEL_DIRECT
    B.conv2d_desc_destroy(d)


def test_split_reduction_plan(monkeypatch):
    """Few output tiles and a long reduction: the implicit path splits the reduction."""
    monkeypatch.delenv("CONV2D_KSPLIT", raising=False)
    def plan(cs):
        d = B.conv2d_desc_create(params_for(cs))
        try:
            return B.conv2d_plan_query(d, B.CONV2D_ALGO_IMPLICIT_GEMM)
        finally:
            B.conv2d_desc_destroy(d)
    small = datagen.CONFIGS["cfg2"].with_(n=1, c=512, h=7, w=7, k=256)   # 4 tiles, 4608-long reduction
    info = plan(small)
    assert info.ksplit > 1 and info.workspace_bytes == info.ksplit * 256 * 49 * 4
    assert plan(datagen.CONFIGS["cfg2"]).ksplit == 1                    # 1568 tiles
    monkeypatch.setenv("CONV2D_KSPLIT", "3")
    assert plan(datagen.CONFIGS["cfg2"]).ksplit == 3


def test_tail_split_plan(monkeypatch):
    """Tile counts a little above a multiple of the 256 CUs: the tiles past it are computed
    in pieces of consecutive stages, so every CU gets the same share of tile work."""
    monkeypatch.delenv("CONV2D_TAIL", raising=False)
    monkeypatch.delenv("CONV2D_KSPLIT", raising=False)

    def plan(cs):
        d = B.conv2d_desc_create(params_for(cs))
        try:
            return B.conv2d_plan_query(d, B.CONV2D_ALGO_IMPLICIT_GEMM)
        finally:
            B.conv2d_desc_destroy(d)
    cfg2 = datagen.CONFIGS["cfg2"]
    info = plan(cfg2)                        # 1568 = 6 * 256 + 32 tiles of 64 x 64, 18 stages of 32
    assert (info.tail_tiles, info.tail_pieces) == (32, 6)           # 8 wanted: pieces of 3 -> 6
    assert info.workspace_bytes == 32 * 6 * 64 * 64 * 4
    assert info.kred_pad == 576
    info = plan(cfg2.with_(n=31))            # 1519 tiles: 239 past 5 * 256, more than half the CUs
    assert info.tail_tiles == 0
    info = plan(cfg2.with_(n=2))             # 98 tiles: fewer than the CUs, no tail
    assert info.tail_tiles == 0
    assert plan(datagen.CONFIGS["cfg3a"]).tail_pieces == 8      # 16 stages: pieces of 2
    assert plan(cfg2.with_(groups=2)).tail_tiles == 0           # one group only
    monkeypatch.setenv("CONV2D_TAIL", "0")
    assert plan(cfg2).tail_tiles == 0
    monkeypatch.setenv("CONV2D_TAIL", "5")
    small = cfg2.with_(n=1, h=13, w=11, k=70)    # 2 x 3 tiles, all computed in 5 pieces
    assert plan(small).ksplit > 1                # (the split reduction comes first)
    monkeypatch.setenv("CONV2D_KSPLIT", "1")
    info = plan(small)
    assert (info.tail_tiles, info.tail_pieces) == (6, 5)
    assert plan(cfg2).tail_pieces == 5


def test_grouped_auto_choice():
    """Grouped layers: few channels per group go to the direct (vector ALU) kernels, wider
    groups to the MFMA implicit path."""
    base = datagen.CONFIGS["cfg2"].with_(c=256, k=256)

    def algo(**kw):
        d = B.conv2d_desc_create(params_for(base.with_(**kw)))
        try:
            return B.conv2d_plan_query(d, B.CONV2D_ALGO_AUTO).algo
        finally:
            B.conv2d_desc_destroy(d)
    assert algo(groups=256) == B.CONV2D_ALGO_DIRECT                  # depthwise
    assert algo(groups=32) == B.CONV2D_ALGO_DIRECT                   # C/g = K/g = 8
    assert algo(groups=16) == B.CONV2D_ALGO_DIRECT                   # 16, 16
    assert algo(groups=8) == B.CONV2D_ALGO_IMPLICIT_GEMM             # 32, 32
    assert algo(groups=16, k=1024) == B.CONV2D_ALGO_IMPLICIT_GEMM    # 16, 64
    assert algo(groups=64, k=2048) == B.CONV2D_ALGO_DIRECT           # 4, 32
    assert algo(groups=1) == B.CONV2D_ALGO_WINOGRAD                  # 256 -> 256, 3x3, stride 1
    # ungrouped, K <= 16: the direct kernel when its grid fills the chip and the filter is not 1x1
    # (for K = 5..16 only with a reduction of at most 256)
    assert algo(c=512, k=3, h=112, w=112) == B.CONV2D_ALGO_DIRECT        # 32 images x 13 bands
    assert algo(c=512, k=16, h=112, w=112) == B.CONV2D_ALGO_IMPLICIT_GEMM  # reduction 4608
    assert algo(c=16, k=16, h=112, w=112) == B.CONV2D_ALGO_DIRECT         # reduction 144
    assert algo(c=512, k=32, h=112, w=112) == B.CONV2D_ALGO_IMPLICIT_GEMM
    # 26 grouped-kernel blocks; K <= 4: the few-output-channel kernel splits the channels instead
    assert algo(n=2, c=512, k=3, h=112, w=112) == B.CONV2D_ALGO_DIRECT
    assert algo(n=2, c=512, k=16, h=112, w=112) == B.CONV2D_ALGO_IMPLICIT_GEMM
    assert algo(c=512, k=3, h=112, w=112, r=1, s=1, pad=(0, 0)) == B.CONV2D_ALGO_IMPLICIT_GEMM


def test_winograd_plan(monkeypatch):
    cfg2 = datagen.CONFIGS["cfg2"]

    def plan(cs):
        d = B.conv2d_desc_create(params_for(cs))
        try:
            return B.conv2d_plan_query(d, B.CONV2D_ALGO_WINOGRAD)
        finally:
            B.conv2d_desc_destroy(d)
    monkeypatch.setenv("CONV2D_WINO_TILE", "4")
    info = plan(cfg2)
    tiles4 = 32 * 14 * 14
    assert info.wino_tile == 4 and info.chunks == 1
    assert info.workspace_bytes == 36 * 64 * 64 * 4 + 36 * (64 + 64) * tiles4 * 4
    assert plan(cfg2.with_(h=57, w=55)).workspace_bytes == 36 * 64 * 64 * 4 + 36 * 128 * 32 * 15 * 14 * 4
    monkeypatch.setenv("CONV2D_WINO_TILE", "2")
    info = plan(cfg2)
    tiles = 32 * 28 * 28
    assert info.algo == B.CONV2D_ALGO_WINOGRAD and info.chunks == 1 and info.kred == 64 and info.wino_tile == 2
    assert info.workspace_bytes == 16 * 64 * 64 * 4 + 16 * (64 + 64) * tiles * 4
    for bad in (cfg2.with_(r=5, s=5, pad=(2, 2)), cfg2.with_(stride=(2, 2)), cfg2.with_(dil=(2, 2), pad=(2, 2)),
                cfg2.with_(groups=2), cfg2.with_(x_dtype="bf16", y_dtype="bf16", c=60)):
        with pytest.raises(B.Conv2dError) as e:
            plan(bad)
        assert e.value.status == B.CONV2D_E_UNSUPPORTED
    def auto(cs):
        d = B.conv2d_desc_create(params_for(cs))
        try:
            return B.conv2d_plan_query(d, B.CONV2D_ALGO_AUTO).algo
        finally:
            B.conv2d_desc_destroy(d)
    assert auto(cfg2) == B.CONV2D_ALGO_IMPLICIT_GEMM                       # 64 channels
    assert auto(cfg2.with_(c=128, k=256)) == B.CONV2D_ALGO_WINOGRAD
    assert auto(cfg2.with_(c=512, k=512, h=7, w=7)) == B.CONV2D_ALGO_WINOGRAD         # 7x7, 7.4 GFLOP
    assert auto(cfg2.with_(n=8, c=512, k=512, h=7, w=7)) == B.CONV2D_ALGO_IMPLICIT_GEMM  # 1.9 GFLOP
    # bf16: F(2x2) only, U and V in bf16, V from the NHWC copy of x; not taken by AUTO
    bf = cfg2.with_(x_dtype="bf16", y_dtype="bf16")
    info = plan(bf)
    tiles2 = 32 * 28 * 28
    assert info.wino_tile == 2 and info.needs_reorder == 1
    assert info.workspace_bytes == 16 * 64 * 64 * 2 + 16 * (64 * 2 + 64 * 4) * tiles2
    assert auto(bf.with_(c=256, k=256)) != B.CONV2D_ALGO_WINOGRAD
    monkeypatch.delenv("CONV2D_WINO_TILE")
    assert plan(cfg2).wino_tile == 4 and plan(cfg2.with_(h=14, w=14)).wino_tile == 4
    assert plan(cfg2.with_(h=7, w=7)).wino_tile == 2 and plan(cfg2.with_(h=40, w=7)).wino_tile == 2
    monkeypatch.setenv("CONV2D_WINO_TILE", "2")
    assert auto(cfg2.with_(c=256, k=256, stride=(2, 2))) == B.CONV2D_ALGO_IMPLICIT_GEMM
    monkeypatch.setenv("CONV2D_WORKSPACE_LIMIT_BYTES", str(64 << 20))
    info = plan(cfg2)
    assert info.chunks == -(-tiles // ((64 << 20) // (16 * 128 * 4)))
    monkeypatch.setenv("CONV2D_WORKSPACE_LIMIT_BYTES", "0")
    with pytest.raises(B.Conv2dError) as e:
        plan(cfg2)
    assert e.value.status == B.CONV2D_E_ALLOC


def test_explicit_workspace_chunking(monkeypatch):
    cs = datagen.CONFIGS["cfg4"]
    d = B.conv2d_desc_create(params_for(cs))
    info = B.conv2d_plan_query(d, B.CONV2D_ALGO_IM2COL_GEMM)
    # col (147 x 401408 fp32) + result (64 x 401408 fp32) fits the 1 GiB default in one chunk
    assert info.chunks == 1 and info.workspace_bytes == 401408 * (147 + 64) * 4
    B.conv2d_desc_destroy(d)
    monkeypatch.setenv("CONV2D_WORKSPACE_LIMIT_BYTES", str(64 << 20))
    d = B.conv2d_desc_create(params_for(cs))
    info = B.conv2d_plan_query(d, B.CONV2D_ALGO_IM2COL_GEMM)
    assert info.chunks > 1 and info.workspace_bytes <= 64 << 20
    B.conv2d_desc_destroy(d)
    monkeypatch.setenv("CONV2D_WORKSPACE_LIMIT_BYTES", "0")
    d = B.conv2d_desc_create(params_for(cs))
    with pytest.raises(B.Conv2dError) as ei:
        B.conv2d_plan_query(d, B.CONV2D_ALGO_IM2COL_GEMM)
    assert ei.value.status == B.CONV2D_E_ALLOC
    B.conv2d_desc_destroy(d)


def test_status_strings():
    for code in range(-8, 1):
        assert isinstance(B.conv2d_status_string(code), str)
        assert B.conv2d_status_string(code) != "unknown status"
    assert "scratch" in B.conv2d_status_string(B.CONV2D_E_SCRATCH)
    assert B.conv2d_status_string(0) == "ok"


def test_bf16_small_group_nhwc_plan(monkeypatch):
    """bf16 with C/g = 8 or 16 gathers whole taps from the NHWC copy (16-byte runs) when the
    layer does enough work per input byte; other small C/g keep the NCHW gathers."""
    for k in ("CONV2D_NHWC_GATHER", "CONV2D_SLICE"):
        monkeypatch.delenv(k, raising=False)
    base = datagen.ConvShape(n=32, c=16, h=56, w=56, k=1024, r=5, s=5, stride=(1, 1), pad=(2, 2), dil=(1, 1),
                             groups=1, seed=1, has_bias=True, x_dtype="bf16", y_dtype="bf16")

    def plan(cs):
        d = B.conv2d_desc_create(params_for(cs))
        try:
            return B.conv2d_plan_query(d, B.CONV2D_ALGO_IMPLICIT_GEMM)
        finally:
            B.conv2d_desc_destroy(d)
    for cs in (base, base.with_(c=8), base.with_(c=64, groups=4)):
        p = plan(cs)
        assert p.kernel == B.CONV2D_KERNEL_GEMM and p.needs_reorder == 1, cs
        assert p.kred_pad == -(-p.kred // 32) * 32
    assert plan(base.with_(c=24)).needs_reorder == 0                  # C/g = 24: NCHW gather
    assert plan(base.with_(x_dtype="f32", y_dtype="f32")).needs_reorder == 0
    assert plan(base.with_(k=16, r=3, s=3, pad=(1, 1))).needs_reorder == 0   # 144 flops per byte
    # NHWC x and y: the gather reads x as it is and the GEMM's epilogue writes NHWC y (bf16, and
    # fp32 with C/g a multiple of 16); fp32 with C/g = 24 reads an NCHW copy and reorders y
    for dt in ("bf16", "f32"):
        p = plan(base.with_(layout="nhwc", x_dtype=dt, y_dtype=dt))
        assert p.kernel == B.CONV2D_KERNEL_GEMM and p.ksplit <= 1 and p.needs_reorder == 0, dt
    assert plan(base.with_(layout="nhwc", c=24, x_dtype="f32", y_dtype="f32")).needs_reorder == 1


def test_depthwise_nhwc_plan(monkeypatch):
    """Depthwise NHWC layers (C a multiple of 4) run the NHWC depthwise kernel without layout
    reorders; C = 6, NCHW and the forced generic kernel keep the reorders or the NCHW kernels."""
    monkeypatch.delenv("CONV2D_DW_GENERIC", raising=False)
    base = datagen.ConvShape(n=2, c=64, h=15, w=17, k=64, r=3, s=3, stride=(1, 1), pad=(1, 1), dil=(1, 1),
                             groups=64, seed=1, has_bias=True, layout="nhwc")

    def plan(cs):
        d = B.conv2d_desc_create(params_for(cs))
        try:
            return B.conv2d_plan_query(d, B.CONV2D_ALGO_DIRECT)
        finally:
            B.conv2d_desc_destroy(d)
    assert plan(base).needs_reorder == 0
    assert plan(base.with_(x_dtype="bf16", y_dtype="bf16")).needs_reorder == 0
    assert plan(base.with_(c=6, k=6, groups=6)).needs_reorder == 1
    assert plan(base.with_(layout="nchw")).needs_reorder == 0
    monkeypatch.setenv("CONV2D_DW_GENERIC", "1")
    assert plan(base).needs_reorder == 1


def test_small_m_tile_choice(monkeypatch):
    """Few output channels per group: the planner takes a 32-row GEMM tile instead of leaving
    most of a 64-row tile idle; 64 or more keep the 64-row tiles."""
    monkeypatch.delenv("CONV2D_GEMM", raising=False)
    base = datagen.ConvShape(n=32, c=512, h=56, w=56, k=16, r=5, s=5, stride=(1, 1), pad=(4, 4), dil=(2, 2),
                             groups=1, seed=1, has_bias=True)

    def tile(cs, algo=B.CONV2D_ALGO_IMPLICIT_GEMM):
        d = B.conv2d_desc_create(params_for(cs))
        try:
            p = B.conv2d_plan_query(d, algo)
            return p.tile_m, p.tile_n
        finally:
            B.conv2d_desc_destroy(d)
    assert tile(base)[0] == 32
    assert tile(base.with_(k=32))[0] == 32
    assert tile(base.with_(k=3))[0] == 32
    assert tile(base, B.CONV2D_ALGO_IM2COL_GEMM)[0] == 32
    assert tile(base.with_(x_dtype="bf16", y_dtype="bf16", k=32))[0] == 32
    assert tile(base.with_(k=64))[0] >= 64
    assert tile(base.with_(k=256))[0] >= 64


def test_smallk_direct_plan(monkeypatch):
    """Ungrouped layers with K <= 4: DIRECT runs the few-output-channel kernel, its input
    channels split into ranges that fill the chip (partials in the workspace)."""
    for k in ("CONV2D_SMALLK", "CONV2D_SMALLK_RANGES", "CONV2D_DW_GENERIC"):
        monkeypatch.delenv(k, raising=False)
    base = datagen.ConvShape(n=8, c=2048, h=112, w=112, k=3, r=7, s=7, stride=(2, 2), pad=(3, 3), dil=(1, 1),
                             groups=1, seed=1, has_bias=True)

    def plan(cs, algo=B.CONV2D_ALGO_DIRECT):
        d = B.conv2d_desc_create(params_for(cs))
        try:
            return B.conv2d_plan_query(d, algo)
        finally:
            B.conv2d_desc_destroy(d)
    p = plan(base)
    P = 8 * 56 * 56
    pblocks = -(-P // 256)
    ranges = min(-(-2048 // pblocks), 2048 // 16)
    assert p.kernel == B.CONV2D_KERNEL_DIRECT and p.ksplit == ranges
    assert p.workspace_bytes == ranges * 3 * P * 4
    assert plan(base.with_(n=16, c=16, h=448, w=448)).ksplit <= 1          # 3136 pixel blocks
    assert plan(base.with_(k=5)).ksplit == 0                                # K > 4: other kernels
    assert plan(base.with_(c=32)).ksplit == 0                               # 32 x 49 < 2048: grouped
    bf = base.with_(x_dtype="bf16", y_dtype="bf16")
    assert plan(bf).ksplit == 0                                             # bf16: other kernels
    assert plan(base, B.CONV2D_ALGO_AUTO).algo == B.CONV2D_ALGO_DIRECT
    assert plan(base.with_(r=1, s=1, pad=(0, 0)), B.CONV2D_ALGO_AUTO).algo != B.CONV2D_ALGO_DIRECT
    monkeypatch.setenv("CONV2D_SMALLK_RANGES", "5")
    assert plan(base).ksplit == 5
    monkeypatch.setenv("CONV2D_SMALLK", "1")
    assert plan(bf).ksplit == 5
    monkeypatch.setenv("CONV2D_SMALLK", "0")
    assert plan(base).ksplit == 0
