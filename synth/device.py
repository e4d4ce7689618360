"""Device-side materialisation of synthetic blocks (see ``synth/__init__.py``)."""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import normal_scale

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libsynth_dev.so")
_lib = None


def build() -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    src = os.path.join(HERE, "synth_dev.hip")
    tmp = LIB + ".tmp"
    subprocess.run([hipcc, "--offload-arch=gfx950", "-O3", "-fPIC", "-shared", "-std=c++17",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                    src, "-o", tmp], check=True, capture_output=True)
    os.replace(tmp, LIB)
    return LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            raise RuntimeError(f"{LIB} is not built; run synth.device.build()")
        _lib = ctypes.CDLL(LIB)
        _lib.synth_fill_normal.restype = ctypes.c_int
        _lib.synth_fill_normal.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                           ctypes.POINTER(ctypes.c_int64),
                                           ctypes.POINTER(ctypes.c_int64), ctypes.c_int64,
                                           ctypes.c_uint64, ctypes.c_float, ctypes.c_void_p]
        _lib.synth_copy.restype = ctypes.c_int
        _lib.synth_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                    ctypes.c_void_p]
    return _lib


def copy_bytes(dst, src, nbytes: int, stream=None):
    """Plain device copy of ``nbytes`` (a multiple of 16) between CUDA tensors."""
    import torch
    assert dst.is_cuda and src.is_cuda and nbytes % 16 == 0
    assert dst.numel() * dst.element_size() >= nbytes <= src.numel() * src.element_size()
    s = stream if stream is not None else torch.cuda.current_stream().cuda_stream
    rc = _load().synth_copy(ctypes.c_void_p(dst.data_ptr()), ctypes.c_void_p(src.data_ptr()),
                            nbytes, ctypes.c_void_p(s))
    if rc != 0:
        raise RuntimeError(f"synth_copy failed ({rc})")


def fill(tensor, key: int, spec_shape, spec_strides, base: int, sigma: float, stream=None):
    """Fill a contiguous CUDA tensor (float32 or bfloat16) of shape ``spec_shape``."""
    import torch
    assert tensor.is_cuda and tensor.is_contiguous()
    assert tuple(tensor.shape) == tuple(spec_shape), (tensor.shape, spec_shape)
    bf16 = {torch.float32: 0, torch.bfloat16: 1}[tensor.dtype]
    nd = len(spec_shape)
    shp = (ctypes.c_int64 * nd)(*spec_shape)
    st = (ctypes.c_int64 * nd)(*spec_strides)
    s = stream if stream is not None else torch.cuda.current_stream().cuda_stream
    rc = _load().synth_fill_normal(ctypes.c_void_p(tensor.data_ptr()), bf16, nd, shp, st, base,
                                   ctypes.c_uint64(key), float(normal_scale(sigma)),
                                   ctypes.c_void_p(s))
    if rc != 0:
        raise RuntimeError(f"synth_fill_normal failed ({rc})")
    return tensor


def materialise(w, spec, device="cuda"):
    """New device tensor holding a described block of workload ``w``."""
    import torch
    st, shape, strides, base, sigma = spec
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    t = torch.empty(shape, dtype=dt, device=device)
    return fill(t, w.key(st), shape, strides, base, sigma)
