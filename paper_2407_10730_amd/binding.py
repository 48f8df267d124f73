"""ctypes binding of libconv2d.so: the C ABI in include/conv2d.h, same names.

Argument marshalling only: every step of the convolution runs in the HIP
library.  Device buffers may be passed as integers (device addresses) or as
objects with a ``data_ptr()`` method (torch tensors); streams as integers or
objects with a ``cuda_stream`` attribute (torch streams).

torch is imported before the library is loaded, so the library's
``libamdhip64.so.7`` dependency binds to the HIP runtime torch already
loaded and both share one runtime instance (streams and pointers agree).
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libconv2d.so")

CONV2D_OK = 0
CONV2D_E_INVALID = -1
CONV2D_E_SHAPE = -2
CONV2D_E_UNSUPPORTED = -3
CONV2D_E_NULL = -4
CONV2D_E_ALLOC = -5
CONV2D_E_HIP = -6
CONV2D_E_NO_DATA = -7
CONV2D_E_SCRATCH = -8
CONV2D_NOALLOC_SCRATCH_BYTES = 64 << 20

CONV2D_NCHW, CONV2D_NHWC = 0, 1
CONV2D_F32, CONV2D_BF16 = 0, 1
CONV2D_ALGO_AUTO, CONV2D_ALGO_IMPLICIT_GEMM, CONV2D_ALGO_IM2COL_GEMM, CONV2D_ALGO_DIRECT = 0, 1, 2, 3
CONV2D_ALGO_WINOGRAD = 4
ALGO_NAMES = {0: "auto", 1: "implicit_gemm", 2: "im2col_gemm", 3: "direct", 4: "winograd"}
PHASE_NAMES = ["pre_analysis", "pre_reorder", "in_tiling", "in_packing", "in_microkernel",
               "in_unpacking", "post_reorder"]
CONV2D_PH_COUNT = 7
CONV2D_TIMING_OFF, CONV2D_TIMING_TOTAL, CONV2D_TIMING_PHASES = 0, 1, 2
CONV2D_KERNEL_GEMM, CONV2D_KERNEL_SLICE, CONV2D_KERNEL_DIRECT = 0, 1, 2
KERNEL_NAMES = {CONV2D_KERNEL_GEMM: "gemm", CONV2D_KERNEL_SLICE: "slice", CONV2D_KERNEL_DIRECT: "direct"}

# every function the header declares
EXPORTS = ("conv2d_desc_create", "conv2d_desc_destroy", "conv2d_output_shape", "conv2d_fwd",
           "conv2d_breakdown", "conv2d_breakdown_reset", "conv2d_set_timing", "conv2d_plan_query",
           "conv2d_status_string", "conv2d_runtime_version", "conv2d_pack_probe", "conv2d_probe_mfma",
           "conv2d_probe_copy", "conv2d_fwd_noalloc", "conv2d_kernel_probe")


class Conv2dError(RuntimeError):
    def __init__(self, status: int, where: str = ""):
        self.status = status
        msg = status_string(status) if _lib is not None else str(status)
        super().__init__(f"{where}: {msg} ({status})" if where else f"{msg} ({status})")


class conv2d_params(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("c", ctypes.c_int64), ("h", ctypes.c_int64),
                ("w", ctypes.c_int64), ("k", ctypes.c_int64), ("r", ctypes.c_int64),
                ("s", ctypes.c_int64),
                ("stride_h", ctypes.c_int32), ("stride_w", ctypes.c_int32),
                ("pad_h", ctypes.c_int32), ("pad_w", ctypes.c_int32),
                ("dil_h", ctypes.c_int32), ("dil_w", ctypes.c_int32), ("groups", ctypes.c_int32),
                ("layout", ctypes.c_int32), ("x_dtype", ctypes.c_int32),
                ("y_dtype", ctypes.c_int32), ("has_bias", ctypes.c_int32)]


class conv2d_breakdown_t(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * CONV2D_PH_COUNT),
                ("calls", ctypes.c_int64 * CONV2D_PH_COUNT),
                ("fused_mask", ctypes.c_uint32), ("algo", ctypes.c_int32),
                ("pack_is_preconv", ctypes.c_int32), ("fwd_calls", ctypes.c_int64),
                ("operation_ms", ctypes.c_double), ("convolution_ms", ctypes.c_double),
                ("total_ms", ctypes.c_double), ("total_calls", ctypes.c_int64)]

    def as_dict(self) -> dict:
        return {
            "algo": ALGO_NAMES.get(self.algo, str(self.algo)),
            "ms": {PHASE_NAMES[i]: self.ms[i] for i in range(CONV2D_PH_COUNT)},
            "calls": {PHASE_NAMES[i]: int(self.calls[i]) for i in range(CONV2D_PH_COUNT)},
            "fused": [PHASE_NAMES[i] for i in range(CONV2D_PH_COUNT) if self.fused_mask >> i & 1],
            "pack_is_preconv": int(self.pack_is_preconv),
            "fwd_calls": int(self.fwd_calls),
            "operation_ms": self.operation_ms,
            "convolution_ms": self.convolution_ms,
            "total_ms": self.total_ms,
            "total_calls": int(self.total_calls),
        }


class conv2d_plan_info(ctypes.Structure):
    _fields_ = [("algo", ctypes.c_int32), ("tile_m", ctypes.c_int32), ("tile_n", ctypes.c_int32),
                ("kred", ctypes.c_int32), ("kred_pad", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_int64), ("chunks", ctypes.c_int64),
                ("needs_reorder", ctypes.c_int32), ("op_class", ctypes.c_int32), ("kernel", ctypes.c_int32),
                ("ksplit", ctypes.c_int32), ("tail_tiles", ctypes.c_int32),
                ("tail_pieces", ctypes.c_int32), ("wino_tile", ctypes.c_int32)]


_lib = None


def load():
    """Load libconv2d.so (after torch).  Raises ImportError if it was never built."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  -- binds the HIP runtime first
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with paper_2407_10730_amd.build.build()")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64p = ctypes.c_void_p, ctypes.c_int, ctypes.POINTER(ctypes.c_int64)
    lib.conv2d_desc_create.argtypes = [ctypes.POINTER(conv2d_params), ctypes.POINTER(vp)]
    lib.conv2d_desc_destroy.argtypes = [vp]
    lib.conv2d_output_shape.argtypes = [vp, i64p]
    lib.conv2d_fwd.argtypes = [vp, vp, vp, vp, vp, i32, vp]
    lib.conv2d_fwd_noalloc.argtypes = [vp, vp, vp, vp, vp, i32, vp]
    lib.conv2d_pack_probe.argtypes = [vp, vp, vp, vp]
    lib.conv2d_kernel_probe.argtypes = [vp, vp, vp, vp, vp, vp]
    lib.conv2d_probe_mfma.argtypes = [i32, ctypes.c_int64, vp, ctypes.c_int64, vp, ctypes.POINTER(ctypes.c_double)]
    lib.conv2d_probe_copy.argtypes = [vp, vp, ctypes.c_int64, vp]
    lib.conv2d_breakdown.argtypes = [vp, i32, ctypes.POINTER(conv2d_breakdown_t)]
    lib.conv2d_breakdown_reset.argtypes = [vp]
    lib.conv2d_set_timing.argtypes = [vp, i32]
    lib.conv2d_plan_query.argtypes = [vp, i32, ctypes.POINTER(conv2d_plan_info)]
    lib.conv2d_status_string.argtypes = [i32]
    lib.conv2d_status_string.restype = ctypes.c_char_p
    lib.conv2d_runtime_version.argtypes = [ctypes.POINTER(ctypes.c_int)]
    for name in EXPORTS:
        if name != "conv2d_status_string":
            getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return int(t.data_ptr())


def _stream(s):
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


def _check(st, where):
    if st != CONV2D_OK:
        raise Conv2dError(st, where)


def status_string(status: int) -> str:
    return load().conv2d_status_string(int(status)).decode()


def conv2d_desc_create(params: conv2d_params) -> int:
    d = ctypes.c_void_p()
    _check(load().conv2d_desc_create(ctypes.byref(params), ctypes.byref(d)), "conv2d_desc_create")
    return d.value


def conv2d_desc_destroy(desc: int) -> None:
    _check(load().conv2d_desc_destroy(desc), "conv2d_desc_destroy")


def conv2d_output_shape(desc: int):
    out = (ctypes.c_int64 * 4)()
    _check(load().conv2d_output_shape(desc, out), "conv2d_output_shape")
    return tuple(int(v) for v in out)


def conv2d_fwd(desc: int, x, w, bias, y, algo: int = CONV2D_ALGO_AUTO, stream=None) -> None:
    _check(load().conv2d_fwd(desc, _ptr(x), _ptr(w), _ptr(bias), _ptr(y), int(algo), _stream(stream)),
           "conv2d_fwd")


def conv2d_fwd_noalloc(desc: int, x, w, bias, y, algo: int = CONV2D_ALGO_AUTO, stream=None) -> None:
    _check(load().conv2d_fwd_noalloc(desc, _ptr(x), _ptr(w), _ptr(bias), _ptr(y), int(algo), _stream(stream)),
           "conv2d_fwd_noalloc")


def conv2d_pack_probe(desc: int, x, w, stream=None) -> None:
    _check(load().conv2d_pack_probe(desc, _ptr(x), _ptr(w), _stream(stream)), "conv2d_pack_probe")


def conv2d_kernel_probe(desc: int, x, w, bias, y, stream=None) -> None:
    _check(load().conv2d_kernel_probe(desc, _ptr(x), _ptr(w), _ptr(bias), _ptr(y), _stream(stream)),
           "conv2d_kernel_probe")


def conv2d_probe_mfma(dtype: int, iters: int, sink, stream=None) -> float:
    """Queue the MFMA issue loop; returns the flops it performs."""
    flops = ctypes.c_double()
    nbytes = sink.numel() * sink.element_size()
    _check(load().conv2d_probe_mfma(int(dtype), int(iters), _ptr(sink), nbytes, _stream(stream),
                                    ctypes.byref(flops)), "conv2d_probe_mfma")
    return flops.value


def conv2d_probe_copy(dst, src, nbytes: int, stream=None) -> None:
    _check(load().conv2d_probe_copy(_ptr(dst), _ptr(src), int(nbytes), _stream(stream)), "conv2d_probe_copy")


def conv2d_breakdown(desc: int, algo: int = CONV2D_ALGO_AUTO) -> conv2d_breakdown_t:
    out = conv2d_breakdown_t()
    _check(load().conv2d_breakdown(desc, int(algo), ctypes.byref(out)), "conv2d_breakdown")
    return out


def conv2d_breakdown_reset(desc: int) -> None:
    _check(load().conv2d_breakdown_reset(desc), "conv2d_breakdown_reset")


def conv2d_set_timing(desc: int, mode: int) -> None:
    _check(load().conv2d_set_timing(desc, int(mode)), "conv2d_set_timing")


def conv2d_plan_query(desc: int, algo: int = CONV2D_ALGO_AUTO) -> conv2d_plan_info:
    out = conv2d_plan_info()
    _check(load().conv2d_plan_query(desc, int(algo), ctypes.byref(out)), "conv2d_plan_query")
    return out


def conv2d_status_string(status: int) -> str:
    return status_string(status)


def conv2d_runtime_version() -> int:
    v = ctypes.c_int()
    _check(load().conv2d_runtime_version(ctypes.byref(v)), "conv2d_runtime_version")
    return v.value
