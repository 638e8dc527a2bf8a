"""Seeded synthetic inputs shared by the oracle-driven tests and the HIP path.

Holds no arithmetic of the method: it maps (seed, stream, index) to numbers with
Philox-4x32-10 (the counter-based generator the paper adopts, Sec. 3) and rounds
them to bf16.  Arrays are returned as numpy ``uint16`` bit patterns (bf16) or
``float32``; callers convert them exactly to float64 (oracle) or upload them to
device memory (HIP path).

Stream ids: ``stream_id(config, layer, tensor)`` = config * 2**16 + layer * 16 + tensor.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "philox_inputs.c")
_LIB = os.path.join(_HERE, "libsynth_inputs.so")

UNIFORM = 0
NORMAL = 1

# tensor slots inside a layer's stream block
T_X, T_W, T_G, T_GAMMA, T_BETA, T_RES, T_DY, T_Y, T_MEAN, T_VAR, T_IDX = range(11)

MASTER_SEED = 0  # the case study starts every run from seed 0 (Sec. 6.1)


def build(force: bool = True) -> str:
    """Compile the generator with gcc (OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11", _SRC, "-o", tmp, "-lm"]
        )
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        lib.synth_philox4x32_10.argtypes = [ctypes.POINTER(ctypes.c_uint32)] * 3
        lib.synth_fill_bf16.argtypes = [
            ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_int,
            ctypes.c_double, ctypes.c_double,
        ]
        lib.synth_fill_f32.argtypes = lib.synth_fill_bf16.argtypes
        lib.synth_indices.argtypes = [
            ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint32,
        ]
        _lib = lib
    return _lib


def stream_id(config: int, layer: int, tensor: int) -> int:
    return (config << 16) + (layer << 4) + tensor


def philox4x32_10(counter, key):
    lib = _load()
    c = (ctypes.c_uint32 * 4)(*counter)
    k = (ctypes.c_uint32 * 2)(*key)
    o = (ctypes.c_uint32 * 4)()
    lib.synth_philox4x32_10(c, k, o)
    return [int(v) for v in o]


def bf16(shape, stream: int, dist: int = NORMAL, p0: float = 0.0, p1: float = 1.0,
         seed: int = MASTER_SEED) -> np.ndarray:
    """bf16 bit patterns (uint16) of the given shape."""
    out = np.empty(shape, dtype=np.uint16)
    _load().synth_fill_bf16(out.ctypes.data, out.size, seed, stream, dist, p0, p1)
    return out


def f32(shape, stream: int, dist: int = NORMAL, p0: float = 0.0, p1: float = 1.0,
        seed: int = MASTER_SEED) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    _load().synth_fill_f32(out.ctypes.data, out.size, seed, stream, dist, p0, p1)
    return out


def indices(count: int, n: int, stream: int, seed: int = MASTER_SEED) -> np.ndarray:
    out = np.empty(count, dtype=np.int64)
    _load().synth_indices(out.ctypes.data, count, n, seed, stream)
    return out


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float64."""
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bf16_bits(v: np.ndarray) -> np.ndarray:
    """Round float64 -> float32 -> bf16 (round to nearest even) bit patterns."""
    u = np.ascontiguousarray(v, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = ((u & 0x7F800000) == 0x7F800000) & ((u & 0x007FFFFF) != 0)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    r = np.where(nan, (u >> 16) | 0x40, r)
    return r.astype(np.uint16)


def kaiming_uniform_bound(fan_in: int) -> float:
    """torch.nn.init.kaiming_uniform_(a=sqrt(5)) bound for a conv weight: 1/sqrt(fan_in)."""
    return 1.0 / float(np.sqrt(fan_in))
