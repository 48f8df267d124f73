"""The measurement entry points on the GPU: the pack probe (the implicit microkernel's
loader alone), the kernel probe (the microkernel alone) and the roofline probes (MFMA
issue loop, device copy)."""
import os

import numpy as np
import pytest

import datagen
from paper_2407_10730_amd import binding as B
from paper_2407_10730_amd.runner import DeviceConv

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load()
    yield
    torch.cuda.synchronize()


def _shape(n, c, h, w, k, r, s, st=(1, 1), pd=(0, 0), dl=(1, 1), g=1, seed=300, dt="f32"):
    return datagen.ConvShape(n=n, c=c, h=h, w=w, k=k, r=r, s=s, stride=st, pad=pd, dil=dl, groups=g, seed=seed,
                             has_bias=True, x_dtype=dt, y_dtype=dt)


# (shape, environment while the descriptor is planned, microkernel expected)
PROBE_CASES = [
    (_shape(2, 32, 13, 11, 70, 3, 3, pd=(1, 1)), {"CONV2D_SLICE": "0"}, B.CONV2D_KERNEL_GEMM),
    (_shape(1, 37, 9, 9, 33, 5, 3, st=(2, 1), pd=(2, 1)), {"CONV2D_SLICE": "0"}, B.CONV2D_KERNEL_GEMM),
    (_shape(2, 3, 24, 224, 64, 7, 7, st=(2, 2), pd=(3, 3)), {"CONV2D_SLICE": "1"}, B.CONV2D_KERNEL_SLICE),
    (_shape(2, 64, 12, 12, 96, 3, 3, pd=(1, 1), dt="bf16"), {"CONV2D_NHWC_GATHER": "1"}, B.CONV2D_KERNEL_GEMM),
    (_shape(1, 96, 6, 7, 40, 3, 3, pd=(1, 1)), {"CONV2D_KSPLIT": "4"}, B.CONV2D_KERNEL_GEMM),
    (_shape(2, 32, 13, 11, 70, 3, 3, pd=(1, 1)), {"CONV2D_TAIL": "3", "CONV2D_KSPLIT": "1"}, B.CONV2D_KERNEL_GEMM),
]


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


@pytest.mark.parametrize("idx", range(len(PROBE_CASES)))
def test_pack_probe_needs_a_call_and_writes_nothing(idx):
    """The probe refuses to run before an implicit call has made its internal copies; after
    one it runs, leaves y untouched, and the next call still gives the same result (the
    loader-only launch leaves no state behind, the tail-split counters included)."""
    import torch
    cs, env, kernel = PROBE_CASES[idx]
    print(f"\n[case] pack probe {cs} env={env}", flush=True)
    with _Env(env):
        dc = DeviceConv(cs, "random")
    try:
        assert dc.plan(B.CONV2D_ALGO_IMPLICIT_GEMM).kernel == kernel
        with pytest.raises(B.Conv2dError) as e:
            B.conv2d_pack_probe(dc.desc, dc.x, dc.w)
        assert e.value.status == B.CONV2D_E_NO_DATA
        dc.run(B.CONV2D_ALGO_IMPLICIT_GEMM)
        torch.cuda.synchronize()
        y0 = dc.y_nchw()
        for _ in range(3):
            B.conv2d_pack_probe(dc.desc, dc.x, dc.w)
        torch.cuda.synchronize()
        assert np.array_equal(dc.y_nchw(), y0)
        dc.y.zero_()
        dc.run(B.CONV2D_ALGO_IMPLICIT_GEMM)
        torch.cuda.synchronize()
        assert np.array_equal(dc.y_nchw(), y0)
    finally:
        dc.close()


@pytest.mark.parametrize("idx", range(len(PROBE_CASES)))
def test_kernel_probe_reproduces_the_microkernel(idx):
    """The kernel probe needs a call first; then, run alone, its microkernel writes the same y
    as the whole call (split-reduction cases: the partials only, y untouched), and calls
    after it still give that result."""
    import torch
    cs, env, kernel = PROBE_CASES[idx]
    print(f"\n[case] kernel probe {cs} env={env}", flush=True)
    with _Env(env):
        dc = DeviceConv(cs, "random")
    try:
        plan = dc.plan(B.CONV2D_ALGO_IMPLICIT_GEMM)
        with pytest.raises(B.Conv2dError) as e:
            B.conv2d_kernel_probe(dc.desc, dc.x, dc.w, dc.b, dc.y)
        assert e.value.status == B.CONV2D_E_NO_DATA
        dc.run(B.CONV2D_ALGO_IMPLICIT_GEMM)
        torch.cuda.synchronize()
        y0 = dc.y.clone()
        dc.y.zero_()
        for _ in range(2):
            B.conv2d_kernel_probe(dc.desc, dc.x, dc.w, dc.b, dc.y)
        torch.cuda.synchronize()
        if plan.ksplit > 1:
            assert not dc.y.any()
        else:
            assert torch.equal(dc.y, y0)
        dc.y.zero_()
        dc.run(B.CONV2D_ALGO_IMPLICIT_GEMM)
        torch.cuda.synchronize()
        assert torch.equal(dc.y, y0)
    finally:
        dc.close()


def test_pack_probe_argument_errors():
    cs = _shape(1, 16, 8, 8, 16, 3, 3, pd=(1, 1))
    dc = DeviceConv(cs, "random")
    try:
        with pytest.raises(B.Conv2dError) as e:
            B.conv2d_pack_probe(dc.desc, None, dc.w)
        assert e.value.status == B.CONV2D_E_NULL
    finally:
        dc.close()


def test_copy_probe_copies():
    import torch
    n = (4 << 20) + 48
    src = torch.randint(0, 255, (n,), dtype=torch.uint8, device="cuda")
    dst = torch.zeros_like(src)
    B.conv2d_probe_copy(dst, src, n)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    for bad in (0, 15, n - 8):
        with pytest.raises(B.Conv2dError) as e:
            B.conv2d_probe_copy(dst, src, bad)
        assert e.value.status == B.CONV2D_E_INVALID


def test_mfma_probe_runs():
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    sink = torch.full((2 * cus * 256,), float("nan"), dtype=torch.float32, device="cuda")
    for dt, per in ((B.CONV2D_F32, 2 * 32 * 32 * 2), (B.CONV2D_BF16, 2 * 32 * 32 * 16)):
        flops = B.conv2d_probe_mfma(dt, 10, sink)
        torch.cuda.synchronize()
        assert flops == 2 * cus * 4 * 4 * 10 * per
        assert bool(torch.isfinite(sink).all())
    with pytest.raises(B.Conv2dError):
        B.conv2d_probe_mfma(B.CONV2D_F32, 0, sink)
    with pytest.raises(B.Conv2dError):
        B.conv2d_probe_mfma(B.CONV2D_F32, 10, sink[:256])
