"""Seeded synthetic inputs for the tree-verification step.

Thin ctypes wrapper over ``gen.c`` plus the workload presets.  Nothing here
computes any part of the verification step itself; the generator only draws
tensors, quantises weights into the int4 storage format, and builds draft
trees and accepted paths.  Both the fp64 reference checker and the GPU path
consume exactly these arrays.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .workloads import CONFIGS, LayerShape, WorkloadConfig, seeds_for  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "_build", "libswiftgen.so")
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    u64, i64, dbl = ctypes.c_uint64, ctypes.c_int64, ctypes.c_double
    vp = ctypes.c_void_p
    lib.gen_normal_f16.argtypes = [u64, u64, u64, i64, dbl, dbl, vp]
    lib.gen_normal_f16.restype = None
    lib.gen_quantize_w4.argtypes = [vp, i64, i64, vp, vp, vp]
    lib.gen_quantize_w4.restype = None
    lib.gen_w4_random.argtypes = [u64, u64, i64, dbl, i64, i64, vp, vp, vp]
    lib.gen_w4_random.restype = None
    lib.gen_tree.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, u64, vp]
    lib.gen_tree.restype = ctypes.c_int
    lib.gen_accept_leaf.argtypes = [vp, ctypes.c_int, u64, ctypes.c_int]
    lib.gen_accept_leaf.restype = ctypes.c_int
    lib.gen_u64.argtypes = [u64, u64, u64, i64, vp]
    lib.gen_u64.restype = None
    lib.gen_f16_from_f64.argtypes = [dbl]
    lib.gen_f16_from_f64.restype = ctypes.c_uint16
    lib.gen_normal_quantile.argtypes = [dbl]
    lib.gen_normal_quantile.restype = dbl
    lib.gen_num_threads.argtypes = []
    lib.gen_num_threads.restype = ctypes.c_int
    _lib = lib
    return lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def normal_f16(seed: int, stream: int, shape, mean: float = 0.0, std: float = 1.0,
               offset: int = 0) -> np.ndarray:
    """fp16 bit patterns (uint16) of N(mean, std) draws, counter-indexed."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    _load().gen_normal_f16(seed, stream, offset, n, mean, std, _ptr(out))
    return out.reshape(shape)


def quantize_w4(w_f16: np.ndarray):
    """Quantise fp16 bits w[N][K] -> (qweight u8[N][K/2], scales u16[N][K/128], zeros u8[N][K/128])."""
    w = np.ascontiguousarray(w_f16, dtype=np.uint16)
    N, K = w.shape
    assert K % 128 == 0
    q = np.empty((N, K // 2), np.uint8)
    s = np.empty((N, K // 128), np.uint16)
    z = np.empty((N, K // 128), np.uint8)
    _load().gen_quantize_w4(_ptr(w), N, K, _ptr(q), _ptr(s), _ptr(z))
    return q, s, z


def w4_random(seed: int, stream: int, N: int, K: int, std: float = 0.02, row0: int = 0,
              nrows: int | None = None):
    """Draw W[N][K] ~ N(0, std) fp16 and quantise it; rows [row0, row0 + nrows)."""
    assert K % 128 == 0
    nrows = N - row0 if nrows is None else nrows
    q = np.empty((nrows, K // 2), np.uint8)
    s = np.empty((nrows, K // 128), np.uint16)
    z = np.empty((nrows, K // 128), np.uint8)
    _load().gen_w4_random(seed, stream, K, std, row0, nrows, _ptr(q), _ptr(s), _ptr(z))
    return q, s, z


def tree(T: int, levels: int, branching: int, seed: int) -> np.ndarray:
    out = np.empty(T, np.int32)
    rc = _load().gen_tree(T, levels, branching, seed, _ptr(out))
    if rc != 0:
        raise ValueError(f"infeasible tree shape T={T} levels={levels} branching={branching}")
    return out


def accept_leaf(parent: np.ndarray, seed: int, deepest_only: bool = False) -> int:
    p = np.ascontiguousarray(parent, dtype=np.int32)
    return int(_load().gen_accept_leaf(_ptr(p), len(p), seed, int(deepest_only)))


def u64(seed: int, stream: int, n: int, offset: int = 0) -> np.ndarray:
    out = np.empty(n, np.uint64)
    _load().gen_u64(seed, stream, offset, n, _ptr(out))
    return out


def num_threads() -> int:
    return int(_load().gen_num_threads())
