"""Runner: one convolution on the GPU through the C ABI, with torch owning memory.

The ConvBench usage pattern (Sec. III-C) is: create the data of an operation
with a data-generation strategy, run the main or the baseline algorithm with
warm-ups and measured runs, and read the timing tool's breakdown.  This
module does the device side of that for one operation: it uploads seeded
inputs (from the ``datagen`` module at the repository root), owns the
descriptor and the output tensor, and launches ``conv2d_fwd``.  No
convolution arithmetic happens here.
"""
from __future__ import annotations

import os
import sys

import numpy as np

from . import binding as B

_ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _datagen():
    if _ROOT not in sys.path:
        sys.path.insert(0, _ROOT)
    import datagen
    return datagen


def params_for(cs) -> B.conv2d_params:
    """conv2d_params of a datagen.ConvShape."""
    return B.conv2d_params(
        n=cs.n, c=cs.c, h=cs.h, w=cs.w, k=cs.k, r=cs.r, s=cs.s,
        stride_h=cs.stride[0], stride_w=cs.stride[1], pad_h=cs.pad[0], pad_w=cs.pad[1],
        dil_h=cs.dil[0], dil_w=cs.dil[1], groups=cs.groups,
        layout=B.CONV2D_NHWC if cs.layout == "nhwc" else B.CONV2D_NCHW,
        x_dtype=B.CONV2D_BF16 if cs.x_dtype == "bf16" else B.CONV2D_F32,
        y_dtype=B.CONV2D_BF16 if cs.y_dtype == "bf16" else B.CONV2D_F32,
        has_bias=1 if cs.has_bias else 0)


def to_device(a: np.ndarray, dtype: str, device):
    """Upload fp32 values as fp32, or as bf16 bit patterns (values must be bf16-exact)."""
    import torch
    if dtype == "bf16":
        dg = _datagen()
        bits = dg.bf16_bits(a)
        if not np.array_equal(dg.bf16_to_f32(bits).reshape(a.shape), a):
            raise ValueError("values are not bf16-exact")
        return torch.from_numpy(bits.view(np.int16).reshape(a.shape)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


def from_device(t) -> np.ndarray:
    """Device tensor (fp32 or bf16) -> float64 numpy array."""
    import torch
    if t.dtype == torch.bfloat16:
        bits = t.view(torch.int16).cpu().numpy().view(np.uint16)
        return _datagen().bf16_to_f32(bits).astype(np.float64).reshape(tuple(t.shape))
    return t.float().cpu().numpy().astype(np.float64)


class DeviceConv:
    """One operation on one device: inputs, descriptor, output."""

    def __init__(self, cs, mode: str = "random", device: str = "cuda:0", inputs=None, device_inputs=None,
                 timing=None):
        """inputs: host float32 (x NCHW, w, b) to upload; device_inputs: tensors already on the
        device in the layout and dtype of `cs` (then x_host etc. are not kept); timing: a
        CONV2D_TIMING_* mode for the descriptor (None keeps the library's default, OFF)."""
        import torch
        self.cs = cs
        self.device = torch.device(device)
        if device_inputs is not None:
            self.x, self.w, self.b = device_inputs
            self.x_host = self.w_host = self.b_host = None
        else:
            if inputs is None:
                inputs = _datagen().make_inputs(cs, mode)
            self.x_host, self.w_host, self.b_host = inputs   # NCHW / KCRS float32 values
            x_dev = self.x_host
            if cs.layout == "nhwc":
                x_dev = np.ascontiguousarray(self.x_host.transpose(0, 2, 3, 1))
            self.x = to_device(x_dev, cs.x_dtype, self.device)
            self.w = to_device(self.w_host, cs.x_dtype, self.device)
            self.b = torch.from_numpy(self.b_host).to(self.device) if cs.has_bias else None
        self.desc = B.conv2d_desc_create(params_for(cs))
        if timing is not None:
            B.conv2d_set_timing(self.desc, timing)
        n, k, ho, wo = B.conv2d_output_shape(self.desc)
        self.out_nkhw = (n, k, ho, wo)
        shape = (n, ho, wo, k) if cs.layout == "nhwc" else (n, k, ho, wo)
        ydt = torch.bfloat16 if cs.y_dtype == "bf16" else torch.float32
        self.y = torch.empty(shape, dtype=ydt, device=self.device)

    def run(self, algo: int = B.CONV2D_ALGO_AUTO, stream=None):
        import torch
        if stream is None:
            stream = torch.cuda.current_stream(self.device)
        B.conv2d_fwd(self.desc, self.x, self.w, self.b, self.y, algo, stream)

    def y_nchw(self) -> np.ndarray:
        y = from_device(self.y)
        if self.cs.layout == "nhwc":
            y = np.ascontiguousarray(y.transpose(0, 3, 1, 2))
        return y

    def breakdown(self, algo: int = B.CONV2D_ALGO_AUTO) -> dict:
        return B.conv2d_breakdown(self.desc, algo).as_dict()

    def plan(self, algo: int = B.CONV2D_ALGO_AUTO):
        return B.conv2d_plan_query(self.desc, algo)

    def close(self):
        if self.desc:
            B.conv2d_desc_destroy(self.desc)
            self.desc = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
