"""The seeded 500-convolution sweep against the point-sampled oracle (needs the GPU).

Shapes follow the sweep rules in datagen.sweep_shapes (fp32 and bf16 alternating, ~20%
depthwise, N in {1, 8, 32}, C, K in 3..2048, H = W in 7..224, 1/3/5/7 filters, stride and
dilation 1 or 2, 'same' padding).  Inputs are generated on the GPU with the same SplitMix64
streams as the host generator.  Every convolution runs with the planner's algorithm; every
tenth also with the explicit im2col path.  Up to 65536 outputs per convolution are checked
(random points plus the corners and one full border row and column of one output plane).
"""
import numpy as np
import pytest

import datagen
import oracle
from paper_2407_10730_amd import binding as B
from paper_2407_10730_amd.runner import DeviceConv

pytestmark = pytest.mark.gpu

CHUNK = 25
COUNT = 500
MAX_POINTS = 65536


def _out_hw(cs):
    return oracle.output_dims(cs.x_shape(), cs.w_shape(), cs.stride, cs.pad, cs.dil, cs.groups)


_SHAPES = None


def _shapes():
    global _SHAPES
    if _SHAPES is None:
        _SHAPES = datagen.sweep_shapes(_out_hw, COUNT)[0]
    return _SHAPES


def sample_points(cs, ho, wo):
    """int64 [npts, 4] rows of (n, k, ho, wo)."""
    total = cs.n * cs.k * ho * wo
    if total <= MAX_POINTS:
        return np.stack(np.unravel_index(np.arange(total), (cs.n, cs.k, ho, wo)), axis=1).astype(np.int64)
    rng = np.random.default_rng(cs.seed)
    n0, k0 = int(rng.integers(cs.n)), int(rng.integers(cs.k))
    edge = [(n0, k0, 0, 0), (n0, k0, 0, wo - 1), (n0, k0, ho - 1, 0), (n0, k0, ho - 1, wo - 1)]
    edge += [(n0, k0, ho - 1, j) for j in range(wo)] + [(n0, k0, i, wo - 1) for i in range(ho)]
    rand = rng.integers(0, total, size=MAX_POINTS - len(edge))
    pts = np.stack(np.unravel_index(rand, (cs.n, cs.k, ho, wo)), axis=1)
    return np.concatenate([np.array(edge, dtype=np.int64), pts.astype(np.int64)])


def _check_one(cs, algos):
    import torch
    dev = torch.device("cuda:0")
    x = datagen.draw_torch(cs.seed, datagen.TENSOR_X, cs.x_shape(), device=dev)
    w = datagen.draw_torch(cs.seed, datagen.TENSOR_W, cs.w_shape(), device=dev)
    b = datagen.draw_torch(cs.seed, datagen.TENSOR_B, (cs.k,), device=dev)
    if cs.x_dtype == "bf16":
        x, w = x.to(torch.bfloat16), w.to(torch.bfloat16)
    ho, wo = _out_hw(cs)
    pts = sample_points(cs, ho, wo)
    pts_dev = torch.from_numpy(pts).to(dev)
    # the oracle reads exactly the values the GPU reads
    xh = x.float().cpu().numpy()
    wh = w.float().cpu().numpy()
    bh = b.cpu().numpy()
    y_ref, a_ref = oracle.conv2d_points(xh, wh, bh, pts, cs.stride, cs.pad, cs.dil, cs.groups)
    gate = 1e-5 if cs.x_dtype == "f32" else 1e-2
    worst = {}
    for algo in algos:
        dc = DeviceConv(cs, device_inputs=(x, w, b))
        try:
            dc.run(algo)
            y = dc.y[pts_dev[:, 0], pts_dev[:, 1], pts_dev[:, 2], pts_dev[:, 3]].float().cpu().numpy()
            torch.cuda.synchronize()
            plan = dc.plan(algo)
        finally:
            dc.close()
        lit, pt = oracle.normalised_errors(y.astype(np.float64), y_ref, a_ref)
        worst[B.ALGO_NAMES[plan.algo]] = pt
        assert pt <= gate, f"{cs} algo {B.ALGO_NAMES[plan.algo]}: per-point error {pt:.3e} > {gate}"
    return worst


@pytest.mark.parametrize("chunk", range(COUNT // CHUNK))
def test_sweep_chunk(chunk):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load()
    for i in range(chunk * CHUNK, (chunk + 1) * CHUNK):
        cs = _shapes()[i]
        algos = [B.CONV2D_ALGO_AUTO] + ([B.CONV2D_ALGO_IM2COL_GEMM] if i % 10 == 0 else [])
        print(f"[sweep {i}] {cs.name} n{cs.n} c{cs.c} {cs.h}x{cs.w} k{cs.k} r{cs.r} s{cs.stride[0]} "
              f"d{cs.dil[0]} g{cs.groups} {cs.x_dtype}", flush=True)
        worst = _check_one(cs, algos)
        print(f"[sweep {i}] ok {worst}", flush=True)
