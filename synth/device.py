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
        _lib.synth_read.restype = ctypes.c_int
        _lib.synth_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int,
                                    ctypes.c_void_p]
        _lib.synth_empty.restype = ctypes.c_int
        _lib.synth_empty.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
        _lib.synth_mfma_loop.restype = ctypes.c_int
        _lib.synth_mfma_loop.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                         ctypes.c_void_p]
    return _lib


def measured_peaks(reps: int = 5):
    """Achievable rates on this device, for fractions beside the spec peaks:
    a streaming read of 4 GiB (past the 256 MB Infinity Cache; the best of a
    few grid sizes) in GB/s, and the dense bf16 MFMA issue rate of register
    operands on every SIMD in TFLOP/s; each the best of ``reps`` timed runs."""
    import torch
    lib = _load()
    stream = torch.cuda.current_stream()
    s = ctypes.c_void_p(stream.cuda_stream)
    nbytes = 4 << 30
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    buf.fill_(1)

    def timed(launch):
        best = None
        launch()
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            launch()
            e1.record(stream)
            e1.synchronize()
            t = e0.elapsed_time(e1) / 1e3
            best = t if best is None else min(best, t)
        return best

    read = 0.0
    for blocks in (1024, 2048, 4096, 8192):
        out = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")

        def launch(blocks=blocks, out=out):
            if lib.synth_read(ctypes.c_void_p(buf.data_ptr()), nbytes, ctypes.c_void_p(out.data_ptr()),
                              blocks, s) != 0:
                raise RuntimeError("synth_read failed")
        read = max(read, nbytes / timed(launch) / 1e9)
    del buf
    blocks, iters = 2048, 2048   # 2 wavefronts per SIMD on 256 CUs
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")

    def mfma():
        if lib.synth_mfma_loop(blocks, iters, ctypes.c_void_p(out.data_ptr()), s) != 0:
            raise RuntimeError("synth_mfma_loop failed")
    flops = blocks * 4 * iters * 8 * 32768.0
    mfma_tf = flops / timed(mfma) / 1e12

    def empties():   # 200 back-to-back launches of an empty 256-workgroup kernel
        for _ in range(200):
            if lib.synth_empty(256, ctypes.c_void_p(out.data_ptr()), s) != 0:
                raise RuntimeError("synth_empty failed")
    launch_us = timed(empties) / 200 * 1e6
    return {"hbm_read_gbs": read, "mfma_bf16_tflops": mfma_tf, "kernel_launch_us": launch_us,
            "method": "best of 5: 4 GiB streaming read (16-byte loads, 1024-8192 workgroups); "
                      "8 chains of v_mfma_f32_32x32x16_bf16 on registers, 8 wavefronts per CU; "
                      "200 back-to-back launches of an empty kernel"}


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
