"""Seeded synthetic inputs for the P-Reduce path (parameters, gradients).

This module is the one piece that both sides of a parity check use: the CPU
oracle's tests and the HIP path's tests/bench draw their inputs from it, so the
two see identical bytes.  It holds none of the method's arithmetic (no update,
no averaging); it only turns (seed, tag, replica, step, element index) into a
number.

Generator (counter-based, so any window of any step can be regenerated alone):

* ``mix64`` is the SplitMix64 output function of Steele, Lea & Flood,
  "Fast splittable pseudorandom number generators" (OOPSLA 2014), in the
  widely published 64-bit form: xor-shift 30 / multiply 0xBF58476D1CE4E5B9,
  xor-shift 27 / multiply 0x94D049BB133111EB, xor-shift 31.  The stream
  increment is the golden-ratio constant GAMMA = 0x9E3779B97F4A7C15; the i-th
  output (i >= 1) of a stream seeded with s is ``mix64(s + i*GAMMA)``.
* A key is folded from components: ``k0 = seed``, ``k_j = mix64(k_{j-1} +
  GAMMA*(c_j + 1))``.  Inputs use ``key(seed, tag, replica, step)``.
* Element e of a keyed stream is ``h = mix64(key + GAMMA*(e + 1))``.
* Normal-like values: Irwin-Hall(4) on the four 16-bit lanes of h,
  ``D = sum_j ((h >> 16 j) & 0xFFFF) - 131070`` (an exact integer in
  [-131070, 131070]), then ``value = fp32(D) * fp32(sigma*sqrt(3)/65536)``
  with the constant formed in float64 and rounded once.  Variance is
  sigma^2 (to 1 part in 2^32), the support is bounded at about +-3.46 sigma.
  Integer work plus one IEEE fp32 multiply: bit-identical on CPU and GPU.
* bf16 storage takes that fp32 value rounded to nearest-even.

The GPU twin lives in ``seedgen/csrc/seedgen.hip`` (``libseedgen.so``); it
implements the same published definition independently of this file.
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
MUL1 = 0xBF58476D1CE4E5B9
MUL2 = 0x94D049BB133111EB
MASK64 = (1 << 64) - 1

TAG_PARAM = 1
TAG_GRAD = 2

DTYPE_F32 = 0
DTYPE_BF16 = 1


def mix64(z: int) -> int:
    """SplitMix64 output function on a Python int (mod 2^64)."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * MUL1) & MASK64
    z = ((z ^ (z >> 27)) * MUL2) & MASK64
    return z ^ (z >> 31)


def key(seed: int, *components: int) -> int:
    """Fold components into a 64-bit stream key (see module docstring)."""
    k = seed & MASK64
    for c in components:
        k = mix64(k + GAMMA * (c + 1))
    return k


def input_key(seed: int, tag: int, replica: int, step: int) -> int:
    return key(seed, tag, replica, step)


def scale_f32(sigma: float) -> np.float32:
    """fp32(sigma*sqrt(3)/65536), formed in float64 and rounded once."""
    return np.float32(sigma * math.sqrt(3.0) / 65536.0)


def _mix64_np(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * np.uint64(MUL1)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(MUL2)
    return z ^ (z >> np.uint64(31))


def hashes(k: int, start: int, count: int) -> np.ndarray:
    """h_e = mix64(k + GAMMA*(e+1)) for e in [start, start+count), uint64."""
    e1 = np.arange(start + 1, start + 1 + count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(k) + e1 * np.uint64(GAMMA)
        return _mix64_np(z)


def irwin_hall_int(h: np.ndarray) -> np.ndarray:
    """D = sum of the four 16-bit lanes of h, minus 131070 (int32)."""
    m = np.uint64(0xFFFF)
    s = (h & m) + ((h >> np.uint64(16)) & m) + ((h >> np.uint64(32)) & m) + (h >> np.uint64(48))
    return s.astype(np.int64).astype(np.int32) - np.int32(131070)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16 bit pattern (uint16); NaN kept quiet."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = ((b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16))
    nan = (b & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
    quiet = (b >> np.uint32(16)) | np.uint32(0x0040)
    return np.where(nan, quiet, rounded).astype(np.uint16)


def normal_f32(seed: int, tag: int, replica: int, step: int, start: int, count: int,
               sigma: float) -> np.ndarray:
    """fp32 values of the keyed stream for elements [start, start+count)."""
    h = hashes(input_key(seed, tag, replica, step), start, count)
    d = irwin_hall_int(h).astype(np.float32)
    return d * scale_f32(sigma)


def normal(seed: int, tag: int, replica: int, step: int, start: int, count: int,
           sigma: float, dtype: int) -> np.ndarray:
    """Stored values: float32 array, or uint16 bf16 bit patterns for bf16."""
    v = normal_f32(seed, tag, replica, step, start, count, sigma)
    if dtype == DTYPE_F32:
        return v
    if dtype == DTYPE_BF16:
        return f32_to_bf16_bits(v)
    raise ValueError(f"unknown dtype {dtype}")


# --------------------------------------------------------------------------
# GPU twin (libseedgen.so).  Loaded lazily; only callers that generate device
# inputs need it.
# --------------------------------------------------------------------------
_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libseedgen.so")
_lib = None


def gpu_lib():
    global _lib
    if _lib is None:
        import torch  # noqa: F401  -- bind to torch's HIP runtime (see the binding)
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(LIB_PATH)
        lib.seedgen_fill_normal.restype = ctypes.c_int32
        lib.seedgen_fill_normal.argtypes = [
            ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_int64,
            ctypes.c_int64, ctypes.c_float, ctypes.c_void_p]
        _lib = lib
    return _lib


def fill_normal_gpu(ptr: int, dtype: int, seed: int, tag: int, replica: int, step: int,
                    start: int, count: int, sigma: float, stream: int) -> None:
    """Write elements [start, start+count) of the keyed stream to device memory
    at ``ptr`` (which holds element ``start`` at offset 0), on ``stream``."""
    rc = gpu_lib().seedgen_fill_normal(
        ctypes.c_void_p(ptr), dtype, input_key(seed, tag, replica, step), start, count,
        float(scale_f32(sigma)), ctypes.c_void_p(stream))
    if rc != 0:
        raise RuntimeError(f"seedgen_fill_normal failed with code {rc}")


def fill_tensor(t, seed: int, tag: int, replica: int, step: int, sigma: float,
                start: int = 0) -> None:
    """Fill a contiguous CUDA tensor (float32 or bfloat16) on torch's current stream."""
    import torch
    assert t.is_cuda and t.is_contiguous()
    dtype = {torch.float32: DTYPE_F32, torch.bfloat16: DTYPE_BF16}[t.dtype]
    fill_normal_gpu(t.data_ptr(), dtype, seed, tag, replica, step, start, t.numel(), sigma,
                    torch.cuda.current_stream(t.device).cuda_stream)
