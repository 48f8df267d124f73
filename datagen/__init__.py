"""Seeded synthetic inputs shared by the tests, the benchmark and the oracle checks.

This module holds no convolution arithmetic: it only draws numbers, rounds
them to the storage type and describes the shapes of the benchmark workloads.
Both the HIP path and the CPU oracle consume the arrays it returns.

Random stream
-------------
Every tensor is drawn from its own SplitMix64 stream (Steele, Lea and Flood,
"Fast splittable pseudorandom number generators", OOPSLA 2014; the 64-bit
finaliser is the one Vigna publishes with splitmix64.c).  The stream for
``(seed, tensor_id)`` starts from ``mix64((seed << 8) | tensor_id)`` with
tensor ids x=0, w=1, bias=2, and element ``i`` of the tensor is
``mix64(start + (i + 1) * GAMMA)``, i.e. the (i+1)-th output of a SplitMix64
generator seeded with ``start``.

* ``random``  : u = (z >> 40) * 2**-24 in [0, 1), value = 2u - 1, so U[-1, 1)
  on a 2**-23 grid; every value is exact in fp32.
* ``integer`` : floor(9u) - 4, integers in [-4, 4] (exact in bf16 and fp32).
* ``constant``: every element equals one given value.

ConvBench fills its buffers either with random or with constant values
(Sec. III-C, the data-generation option of ``convset_exec``); the integer mode
is an addition for bit-exact GPU checks.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from typing import Optional

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
_M1 = 0xBF58476D1CE4E5B9
_M2 = 0x94D049BB133111EB
_MASK = (1 << 64) - 1

TENSOR_X, TENSOR_W, TENSOR_B = 0, 1, 2


def mix64_int(z: int) -> int:
    """SplitMix64 output finaliser on a Python int (reference for the vector form)."""
    z &= _MASK
    z = ((z ^ (z >> 30)) * _M1) & _MASK
    z = ((z ^ (z >> 27)) * _M2) & _MASK
    return z ^ (z >> 31)


def splitmix64_int(state: int, count: int) -> list[int]:
    """First ``count`` outputs of a SplitMix64 generator seeded with ``state``."""
    out = []
    for _ in range(count):
        state = (state + GAMMA) & _MASK
        out.append(mix64_int(state))
    return out


def _mix64_vec(z: np.ndarray) -> np.ndarray:
    z = z.copy()
    z ^= z >> np.uint64(30)
    z *= np.uint64(_M1)
    z ^= z >> np.uint64(27)
    z *= np.uint64(_M2)
    z ^= z >> np.uint64(31)
    return z


def stream_start(seed: int, tensor_id: int) -> int:
    if not (0 <= seed < (1 << 56)) or not (0 <= tensor_id < 256):
        raise ValueError("seed must be in [0, 2**56) and tensor_id in [0, 256)")
    return mix64_int((seed << 8) | tensor_id)


def raw_stream(seed: int, tensor_id: int, count: int, chunk: int = 1 << 22) -> np.ndarray:
    """``count`` uint64 draws of the (seed, tensor_id) stream."""
    start = np.uint64(stream_start(seed, tensor_id))
    out = np.empty(count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        for lo in range(0, count, chunk):
            hi = min(count, lo + chunk)
            i = np.arange(lo + 1, hi + 1, dtype=np.uint64)
            out[lo:hi] = _mix64_vec(start + i * np.uint64(GAMMA))
    return out


def uniform01(seed: int, tensor_id: int, count: int) -> np.ndarray:
    """u = (z >> 40) * 2**-24, returned as float64 (exact)."""
    z = raw_stream(seed, tensor_id, count)
    return (z >> np.uint64(40)).astype(np.float64) * (2.0 ** -24)


def draw(seed: int, tensor_id: int, shape, mode: str = "random", const: float = 1.0,
         scale: float = 1.0) -> np.ndarray:
    """Draw one tensor as float32 values (fp32-exact; scaled in fp64 then rounded RNE)."""
    count = int(np.prod(shape)) if len(shape) else 1
    if mode == "random":
        v = 2.0 * uniform01(seed, tensor_id, count) - 1.0
    elif mode == "integer":
        v = np.floor(9.0 * uniform01(seed, tensor_id, count)) - 4.0
    elif mode == "constant":
        v = np.full(count, float(const), dtype=np.float64)
    else:
        raise ValueError(f"unknown data mode {mode!r}")
    if scale != 1.0:
        v = v * scale
    return v.astype(np.float32).reshape(shape)


# ---------------------------------------------------------------- bf16 storage

def bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even.  Inputs must be finite."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return rounded.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """fp32 values rounded (RNE) to the nearest bf16, returned as fp32."""
    return bf16_to_f32(bf16_bits(a)).reshape(np.shape(a))


# ---------------------------------------------------------------- workloads

LAYOUTS = {"nchw": 0, "nhwc": 1}
DTYPES = {"f32": 0, "bf16": 1}


@dataclass(frozen=True)
class ConvShape:
    """One conv2d operation: x is N x C x H x W, w is K x C/g x R x S."""
    n: int
    c: int
    h: int
    w: int
    k: int
    r: int
    s: int
    stride: tuple = (1, 1)
    pad: tuple = (0, 0)
    dil: tuple = (1, 1)
    groups: int = 1
    has_bias: bool = True
    layout: str = "nchw"
    x_dtype: str = "f32"
    y_dtype: str = "f32"
    seed: int = 0
    w_scale: Optional[float] = None   # None: weights U[-1,1]; else multiply by this
    name: str = ""

    def with_(self, **kw) -> "ConvShape":
        return replace(self, **kw)

    @property
    def cg(self) -> int:
        return self.c // self.groups

    def x_shape(self):
        return (self.n, self.c, self.h, self.w)

    def w_shape(self):
        return (self.k, self.c // self.groups, self.r, self.s)


def make_inputs(cs: ConvShape, mode: str = "random", const=(1.0, 1.0, 0.0)):
    """x, w, b as float32 arrays in NCHW / KCRS order holding the exact values the
    GPU will read (already rounded to bf16 when x_dtype is bf16).  b is fp32."""
    x = draw(cs.seed, TENSOR_X, cs.x_shape(), mode, const=const[0])
    scale = 1.0 if cs.w_scale is None else cs.w_scale
    w = draw(cs.seed, TENSOR_W, cs.w_shape(), mode, const=const[1], scale=scale)
    if cs.has_bias:
        b = draw(cs.seed, TENSOR_B, (cs.k,), mode, const=const[2])
    else:
        b = np.zeros((cs.k,), dtype=np.float32)
    if cs.x_dtype == "bf16":
        x = round_bf16(x)
        w = round_bf16(w)
    return x, w, b


def _cfg(name, **kw):
    return ConvShape(name=name, **kw)


# The fixed workloads.  Sizes follow the benchmark configurations; seeds are fixed.
CONFIGS = {
    # single small fp32 conv, batch 1 (the paper's protocol is batch 1, Sec. IV)
    "cfg1": _cfg("cfg1", n=1, c=3, h=32, w=32, k=16, r=3, s=3, pad=(1, 1), seed=0),
    # square-channel 3x3 layer, weights scaled by 1/sqrt(C*R*S) = 1/24
    "cfg2": _cfg("cfg2", n=32, c=64, h=56, w=56, k=64, r=3, s=3, pad=(1, 1), seed=2,
                 w_scale=1.0 / math.sqrt(64 * 3 * 3)),
    # pointwise 256 -> 64
    "cfg3a": _cfg("cfg3a", n=32, c=256, h=56, w=56, k=64, r=1, s=1, seed=3),
    # strided pointwise downsample 256 -> 512, stride 2
    "cfg3b": _cfg("cfg3b", n=32, c=256, h=56, w=56, k=512, r=1, s=1, stride=(2, 2), seed=4),
    # low-channel 7x7 stride-2 stem
    "cfg4": _cfg("cfg4", n=32, c=3, h=224, w=224, k=64, r=7, s=7, stride=(2, 2), pad=(3, 3),
                 seed=5),
    "cfg4_bf16": _cfg("cfg4_bf16", n=32, c=3, h=224, w=224, k=64, r=7, s=7, stride=(2, 2),
                      pad=(3, 3), seed=5, x_dtype="bf16", y_dtype="bf16"),
    # a depthwise layer of the sweep's kind (g = C = K), memory bound
    "dw": _cfg("dw", n=32, c=256, h=56, w=56, k=256, r=3, s=3, pad=(1, 1), groups=256, seed=6),
    "dw_bf16": _cfg("dw_bf16", n=32, c=256, h=56, w=56, k=256, r=3, s=3, pad=(1, 1), groups=256, seed=6,
                    x_dtype="bf16", y_dtype="bf16"),
    # grouped layers with 1 < g < C (4 and 8 channels per group), memory bound
    "grp_g64": _cfg("grp_g64", n=32, c=256, h=56, w=56, k=256, r=3, s=3, pad=(1, 1), groups=64, seed=7),
    "grp_g32": _cfg("grp_g32", n=32, c=256, h=56, w=56, k=256, r=3, s=3, pad=(1, 1), groups=32, seed=8),
    # a bf16 layer above the bf16 ridge point (arithmetic intensity ~1100 flop/byte)
    "bf16_3x3": _cfg("bf16_3x3", n=32, c=256, h=56, w=56, k=256, r=3, s=3, pad=(1, 1), seed=9,
                     x_dtype="bf16", y_dtype="bf16"),
}



# ---------------------------------------------------------------- device-side generation

def _i64(v: int) -> int:
    """A 64-bit pattern as a signed int64 value (torch has no uint64 arithmetic)."""
    v &= _MASK
    return v - (1 << 64) if v >= (1 << 63) else v


def _lsr(z, k: int):
    """Logical right shift of int64 bit patterns."""
    return (z >> k) & ((1 << (64 - k)) - 1)


def raw_stream_torch(seed: int, tensor_id: int, count: int, device="cpu", chunk: int = 1 << 26):
    """The uint64 stream of raw_stream() as int64 bit patterns, computed with torch on
    `device` (wrapping int64 arithmetic gives the same bits as uint64)."""
    import torch
    start = _i64(stream_start(seed, tensor_id))
    gamma, m1, m2 = _i64(GAMMA), _i64(_M1), _i64(_M2)
    out = torch.empty(count, dtype=torch.int64, device=device)
    for lo in range(0, count, chunk):
        hi = min(count, lo + chunk)
        z = torch.arange(lo + 1, hi + 1, dtype=torch.int64, device=device) * gamma + start
        z = (z ^ _lsr(z, 30)) * m1
        z = (z ^ _lsr(z, 27)) * m2
        out[lo:hi] = z ^ _lsr(z, 31)
    return out


def draw_torch(seed: int, tensor_id: int, shape, mode: str = "random", const: float = 1.0,
               scale: float = 1.0, device="cpu"):
    """draw() computed on a torch device; returns float32 values bit-identical to draw()."""
    import torch
    count = 1
    for d in shape:
        count *= int(d)
    if mode == "constant":
        v = torch.full((count,), float(const), dtype=torch.float64, device=device)
    else:
        z = raw_stream_torch(seed, tensor_id, count, device)
        u = _lsr(z, 40).to(torch.float64) * (2.0 ** -24)
        del z
        if mode == "random":
            v = 2.0 * u - 1.0
        elif mode == "integer":
            v = torch.floor(9.0 * u) - 4.0
        else:
            raise ValueError(f"unknown data mode {mode!r}")
    if scale != 1.0:
        v = v * scale
    return v.to(torch.float32).reshape(tuple(shape))


def round_bf16_torch(t):
    """Round fp32 values to bf16 (RNE) on the tensor's device; returns torch.bfloat16."""
    import torch
    return t.to(torch.bfloat16)


# ---------------------------------------------------------------- the random sweep

SWEEP_CHANNELS = (3, 16, 32, 64, 128, 256, 512, 1024, 2048)
SWEEP_SIZES = (7, 14, 28, 56, 112, 224)


def sweep_shapes(out_hw, count: int = 500, master_seed: int = 1000, max_bytes: int = 2 << 30,
                 max_flops: float = 2e13):
    """The seeded random sweep of convolutions.

    Draw i (in order): dtype fp32 for even i and bf16 for odd i (y in the same type);
    depthwise with probability 0.2 (then K = C = groups); N in {1, 8, 32}; C and K in
    SWEEP_CHANNELS; H = W in SWEEP_SIZES; R = S in {1, 3, 5, 7}; stride in {1, 2};
    dilation in {1, 2}; 'same' padding p = d*(R-1)/2.  A draw whose fp32 |x| + |y| exceeds
    max_bytes or whose FLOP count exceeds max_flops is rejected and redrawn.  Input seed of
    convolution i is master_seed + i.  `out_hw(shape) -> (Ho, Wo)` is supplied by the caller
    (this module holds no convolution arithmetic).  Returns (shapes, rejected_count).
    """
    rng = np.random.default_rng(master_seed)
    shapes, rejected = [], 0
    while len(shapes) < count:
        i = len(shapes)
        dw = bool(rng.random() < 0.2)
        n = int(rng.choice((1, 8, 32)))
        c = int(rng.choice(SWEEP_CHANNELS))
        k = c if dw else int(rng.choice(SWEEP_CHANNELS))
        h = int(rng.choice(SWEEP_SIZES))
        r = int(rng.choice((1, 3, 5, 7)))
        st = int(rng.choice((1, 2)))
        dl = int(rng.choice((1, 2)))
        p = dl * (r - 1) // 2
        dt = "f32" if i % 2 == 0 else "bf16"
        cs = ConvShape(n=n, c=c, h=h, w=h, k=k, r=r, s=r, stride=(st, st), pad=(p, p), dil=(dl, dl),
                       groups=c if dw else 1, x_dtype=dt, y_dtype=dt, seed=master_seed + i,
                       name=f"sweep{i:03d}")
        ho, wo = out_hw(cs)
        xy = 4 * (n * c * h * h + n * k * ho * wo)
        fl = 2.0 * n * k * (c // cs.groups) * r * r * ho * wo
        if xy > max_bytes or fl > max_flops:
            rejected += 1
            continue
        shapes.append(cs)
    return shapes, rejected
