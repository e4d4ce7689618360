"""Seeded, counter-based synthetic inputs shared by the oracle and the HIP path.

This module holds no arithmetic of the drafter step itself: it only turns
(seed, stream, index) triples into numbers.  Every tensor element is a pure
function of its logical index, so any slice of any tensor can be regenerated
on the host (numpy, here) or on the device (``synth_dev.hip``) with bit-identical
results.

Generator: SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
number generators", OOPSLA 2014), used in counter mode: draw ``i`` of a stream
with key ``k`` is ``mix64(k + (i + 1) * GAMMA)``, where ``mix64`` is the
SplitMix64 output function (Stafford's variant 13).

Distributions built on one 64-bit draw ``z``:

* ``normal``: Irwin-Hall sum of the four 16-bit fields of ``z``, centred and
  scaled to the requested standard deviation.  It has mean 0, the requested
  variance, support of +-3.46 sigma and excess kurtosis -0.3; it stands in
  for N(0, sigma^2).  The final scaling is one IEEE fp32 multiply by a
  constant, so host and device agree bit for bit; bf16 values are the
  round-to-nearest-even of that fp32 value.
* ``uniform_int(lo, hi)``: multiply-shift of the high 32 bits (Lemire 2019).
* ``bernoulli(p)``: high 32 bits compared with round(p * 2^32).
"""
from __future__ import annotations

import math

import numpy as np

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
_M1 = 0xBF58476D1CE4E5B9
_M2 = 0x94D049BB133111EB

# std of the sum of four independent uniforms on {0..65535}
IRWIN_HALL4_STD = math.sqrt((65536.0 ** 2 - 1.0) / 3.0)
IRWIN_HALL4_CENTER = 2 * 65535


def mix64_int(x: int) -> int:
    """SplitMix64 output function on a Python int (scalar keys)."""
    z = x & MASK64
    z = ((z ^ (z >> 30)) * _M1) & MASK64
    z = ((z ^ (z >> 27)) * _M2) & MASK64
    return z ^ (z >> 31)


def stream_key(seed: int, stream: int) -> int:
    """64-bit key of one named sub-stream of a seed."""
    return mix64_int((seed & MASK64) ^ mix64_int((stream + 1) * GAMMA))


def _mix64_np(z: np.ndarray) -> np.ndarray:
    z = z.copy()
    z ^= z >> np.uint64(30)
    z *= np.uint64(_M1)
    z ^= z >> np.uint64(27)
    z *= np.uint64(_M2)
    z ^= z >> np.uint64(31)
    return z


def draw_u64(key: int, idx) -> np.ndarray:
    """Counter-mode SplitMix64 draw for every index in ``idx`` (int64 array)."""
    i = np.asarray(idx, dtype=np.int64).astype(np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(key) + (i + np.uint64(1)) * np.uint64(GAMMA)
    return _mix64_np(z)


def normal_scale(sigma: float) -> np.float32:
    """fp32 constant that maps a centred Irwin-Hall sum to std ``sigma``."""
    return np.float32(sigma / IRWIN_HALL4_STD)


def normal_f32(key: int, idx, sigma: float) -> np.ndarray:
    z = draw_u64(key, idx)
    m = np.uint64(0xFFFF)
    s = ((z & m) + ((z >> np.uint64(16)) & m) + ((z >> np.uint64(32)) & m)
         + (z >> np.uint64(48))).astype(np.int64) - IRWIN_HALL4_CENTER
    return s.astype(np.float32) * normal_scale(sigma)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16, returned as raw uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(u: np.ndarray) -> np.ndarray:
    return (np.asarray(u, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal(key: int, idx, sigma: float, dtype: str) -> np.ndarray:
    """N(0, sigma^2) stand-in; ``dtype`` 'f32' -> float32, 'bf16' -> uint16 bits."""
    f = normal_f32(key, idx, sigma)
    if dtype == "f32":
        return f
    if dtype == "bf16":
        return f32_to_bf16_bits(f)
    raise ValueError(dtype)


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored values (fp32 or bf16 bits) to float64."""
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    return bf16_bits_to_f32(a).astype(np.float64)


def uniform_int(key: int, idx, lo: int, hi: int) -> np.ndarray:
    """Integers uniform on [lo, hi] (inclusive)."""
    z = draw_u64(key, idx) >> np.uint64(32)
    span = np.uint64(hi - lo + 1)
    return (lo + ((z * span) >> np.uint64(32)).astype(np.int64)).astype(np.int64)


def bernoulli(key: int, idx, p: float) -> np.ndarray:
    thr = np.uint64(min(int(round(p * 2.0 ** 32)), 2 ** 32))
    return (draw_u64(key, idx) >> np.uint64(32)) < thr


_HOST_LIB = None


def host_lib():
    """The C build of ``normal`` over a dense block (``synth_host.c``), or None."""
    global _HOST_LIB
    if _HOST_LIB is None:
        import ctypes
        import os
        path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsynth_host.so")
        if not os.path.exists(path):
            return None
        lib = ctypes.CDLL(path)
        lib.synth_host_fill.restype = ctypes.c_int
        lib.synth_host_fill.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                        ctypes.POINTER(ctypes.c_int64),
                                        ctypes.POINTER(ctypes.c_int64), ctypes.c_int64,
                                        ctypes.c_uint64, ctypes.c_float]
        _HOST_LIB = lib
    return _HOST_LIB


def build_host() -> str:
    """Compile synth_host.c into libsynth_host.so next to it."""
    import os
    import subprocess
    here = os.path.dirname(os.path.abspath(__file__))
    out = os.path.join(here, "libsynth_host.so")
    subprocess.run(["gcc", "-O3", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                    os.path.join(here, "synth_host.c"), "-o", out + ".tmp"], check=True)
    os.replace(out + ".tmp", out)
    return out


def normal_block(key: int, shape, strides, base: int, sigma: float, dtype: str,
                 use_c: bool = True) -> np.ndarray:
    """``normal`` over a dense block (logical index base + sum coord * stride),
    through the C build when present, else numpy; both give identical bits.
    dtype 'bf16_f32': the bf16 values, widened exactly to float32."""
    lib = host_lib() if use_c else None
    if lib is None:
        if dtype == "bf16_f32":
            return bf16_bits_to_f32(normal(key, grid_index(shape, strides, base), sigma, "bf16"))
        return normal(key, grid_index(shape, strides, base), sigma, dtype)
    import ctypes
    mode = {"f32": 0, "bf16": 1, "bf16_f32": 2}[dtype]
    out = np.empty(tuple(shape), dtype=np.uint16 if mode == 1 else np.float32)
    nd = len(shape)
    rc = lib.synth_host_fill(out.ctypes.data_as(ctypes.c_void_p), mode, nd,
                             (ctypes.c_int64 * nd)(*shape), (ctypes.c_int64 * nd)(*strides),
                             int(base), ctypes.c_uint64(key), float(normal_scale(sigma)))
    if rc != 0:
        raise RuntimeError("synth_host_fill failed")
    return out


def grid_index(shape, strides, base: int = 0) -> np.ndarray:
    """Flat logical indices of a dense block: base + sum_k coord_k * strides_k."""
    idx = np.full(tuple(shape), base, dtype=np.int64)
    for axis, (n, st) in enumerate(zip(shape, strides)):
        view = [1] * len(shape)
        view[axis] = n
        idx = idx + (np.arange(n, dtype=np.int64) * st).reshape(view)
    return idx
