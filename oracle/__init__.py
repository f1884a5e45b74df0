"""fp64 reference checker for the tree-verification step -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports it and shares no code with it.

numpy wrappers over ``oracle.c``: arrays of fp16 values are uint16 bit
patterns; every function works on host memory only.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "_build", "liboracle.so")
_lib = None

i32, i64, u16, dbl, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint16, ctypes.c_double, ctypes.c_void_p


class Dims(ctypes.Structure):
    _fields_ = [("H", i32), ("Hq", i32), ("Hkv", i32), ("D", i32), ("F", i32), ("S_max", i32),
                ("eps", dbl), ("rope_theta", dbl)]


class W4(ctypes.Structure):
    _fields_ = [("q", vp), ("s", vp), ("z", vp)]


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.oracle_f16_to_f64.argtypes = [u16]
    lib.oracle_f16_to_f64.restype = dbl
    lib.oracle_f64_to_f16.argtypes = [dbl]
    lib.oracle_f64_to_f16.restype = u16
    lib.oracle_tree.argtypes = [vp, i32, vp, vp]
    lib.oracle_tree.restype = ctypes.c_int
    lib.oracle_dequant.argtypes = [vp, vp, vp, i32, i32, i32]
    lib.oracle_dequant.restype = dbl
    lib.oracle_w4a16_gemm.argtypes = [vp, vp, vp, i32, i32, vp, i32, i32, vp, i32, vp, i32]
    lib.oracle_w4a16_gemm.restype = ctypes.c_int
    lib.oracle_w4a16_swiglu.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, vp, i32, i32, vp, i32]
    lib.oracle_w4a16_swiglu.restype = ctypes.c_int
    lib.oracle_rmsnorm.argtypes = [vp, i32, i32, i32, vp, dbl, vp, i32]
    lib.oracle_rmsnorm.restype = ctypes.c_int
    lib.oracle_rope.argtypes = [vp, i32, i64, dbl]
    lib.oracle_rope.restype = None
    lib.oracle_tree_attention.argtypes = [vp, i32, vp, vp, i32, vp, vp, i32, i32, vp, i32, i32,
                                          i32, i32, dbl, dbl, vp, i32]
    lib.oracle_tree_attention.restype = ctypes.c_int
    lib.oracle_kv_commit.argtypes = [vp, vp, i32, i64, i32, i32, i32, i32, vp, i32, i32]
    lib.oracle_kv_commit.restype = i32
    lib.oracle_verify_layer.argtypes = [ctypes.POINTER(Dims), vp, vp, W4, W4, W4, W4, W4, vp, vp,
                                        vp, i32, i32, vp]
    lib.oracle_verify_layer.restype = ctypes.c_int
    lib.oracle_lm_head.argtypes = [vp, i32, i32, vp, dbl, vp, i32, vp]
    lib.oracle_lm_head.restype = ctypes.c_int
    lib.oracle_draft_tree_attention.argtypes = [vp, i32, vp, vp, i32, vp, vp, i32, i32, vp, i32, vp, i32, i32,
                                                i32, i32, dbl, dbl, vp, i32]
    lib.oracle_draft_tree_attention.restype = ctypes.c_int
    lib.oracle_kv_reorganize.argtypes = [vp, vp, i32, i64, i32, i32, i32, i32, vp, i32, i32, i32, vp, vp]
    lib.oracle_kv_reorganize.restype = i32
    lib.oracle_greedy_accept.argtypes = [vp, i32, i32, i32, vp, vp, vp, vp, vp]
    lib.oracle_greedy_accept.restype = i32
    lib.oracle_topk_logprobs.argtypes = [vp, i32, i32, i32, i32, vp, vp]
    lib.oracle_topk_logprobs.restype = i32
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_num_threads.restype = None
    _lib = lib
    return lib


def _p(a):
    if a is None:
        return None
    assert isinstance(a, np.ndarray) and a.flags["C_CONTIGUOUS"], "need C-contiguous numpy array"
    return a.ctypes.data


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def f16_to_f64(h: int) -> float:
    return float(_load().oracle_f16_to_f64(int(h)))


def f64_to_f16(x: float) -> int:
    return int(_load().oracle_f64_to_f16(float(x)))


def f16_array_to_f64(a: np.ndarray) -> np.ndarray:
    f = np.vectorize(lambda h: _load().oracle_f16_to_f64(int(h)), otypes=[np.float64])
    return f(a)


def f64_array_to_f16(a: np.ndarray) -> np.ndarray:
    f = np.vectorize(lambda x: _load().oracle_f64_to_f16(float(x)), otypes=[np.uint16])
    return f(a)


def tree(parent):
    """(depth int32[T], anc uint8[T][T]); raises ValueError on an invalid parent array."""
    p = _c(parent, np.int32)
    T = len(p)
    depth = np.empty(T, np.int32)
    anc = np.empty((T, T), np.uint8)
    if _load().oracle_tree(_p(p), T, _p(depth), _p(anc)) != 0:
        raise ValueError("invalid parent array")
    return depth, anc


def tree_valid(parent) -> bool:
    p = _c(parent, np.int32)
    return _load().oracle_tree(_p(p), len(p), None, None) == 0


def dequant(W: dict, n: int, k: int) -> float:
    return float(_load().oracle_dequant(_p(W["qweight"]), _p(W["scales"]), _p(W["zeros"]),
                                        W["K"], n, k))


def w4a16_gemm(W: dict, x: np.ndarray, residual: np.ndarray | None = None) -> np.ndarray:
    x = _c(x, np.uint16)
    M, K = x.shape
    assert K == W["K"]
    N = W["N"]
    y = np.empty((M, N), np.uint16)
    r = None if residual is None else _c(residual, np.uint16)
    rc = _load().oracle_w4a16_gemm(_p(W["qweight"]), _p(W["scales"]), _p(W["zeros"]), K, N,
                                   _p(x), M, K, _p(r), N, _p(y), N)
    if rc != 0:
        raise ValueError("oracle_w4a16_gemm: invalid arguments")
    return y


def w4a16_swiglu(Wg: dict, Wu: dict, x: np.ndarray) -> np.ndarray:
    x = _c(x, np.uint16)
    M, K = x.shape
    N = Wg["N"]
    y = np.empty((M, N), np.uint16)
    rc = _load().oracle_w4a16_swiglu(_p(Wg["qweight"]), _p(Wg["scales"]), _p(Wg["zeros"]),
                                     _p(Wu["qweight"]), _p(Wu["scales"]), _p(Wu["zeros"]), K, N,
                                     _p(x), M, K, _p(y), N)
    if rc != 0:
        raise ValueError("oracle_w4a16_swiglu: invalid arguments")
    return y


def rmsnorm(x: np.ndarray, gamma: np.ndarray, eps: float = 1e-5) -> np.ndarray:
    x = _c(x, np.uint16)
    M, H = x.shape
    g = _c(gamma, np.uint16)
    out = np.empty((M, H), np.uint16)
    rc = _load().oracle_rmsnorm(_p(x), M, H, H, _p(g), eps, _p(out), H)
    if rc != 0:
        raise ValueError("oracle_rmsnorm: invalid arguments")
    return out


def rope(vec: np.ndarray, pos: int, theta: float = 500000.0) -> np.ndarray:
    v = np.array(vec, dtype=np.float64, copy=True)
    _load().oracle_rope(_p(v), len(v), int(pos), theta)
    return v


def tree_attention(q, k, v, k_cache, v_cache, P, parent, Hq, Hkv, D, rope_theta=500000.0,
                   softmax_scale=None):
    """Returns out [T][Hq*D]; k_cache / v_cache ([Hkv][S_max][D]) are updated in place."""
    q = _c(q, np.uint16)
    k = _c(k, np.uint16)
    v = _c(v, np.uint16)
    p = _c(parent, np.int32)
    T = len(p)
    assert k_cache.flags["C_CONTIGUOUS"] and v_cache.flags["C_CONTIGUOUS"]
    S_max = k_cache.shape[1]
    if softmax_scale is None:
        softmax_scale = 1.0 / np.sqrt(D)
    out = np.empty((T, Hq * D), np.uint16)
    rc = _load().oracle_tree_attention(_p(q), q.shape[1], _p(k), _p(v), k.shape[1], _p(k_cache),
                                       _p(v_cache), S_max, P, _p(p), T, Hq, Hkv, D, rope_theta,
                                       softmax_scale, _p(out), Hq * D)
    if rc != 0:
        raise ValueError("oracle_tree_attention: invalid arguments or tree")
    return out


def draft_tree_attention(q, k, v, k_cache, v_cache, P, cache_parent, leaf_parent, Hq, Hkv, D,
                         rope_theta=500000.0, softmax_scale=None):
    """Draft-model attention with the non-square mask; caches [Hkv][S_max][D]
    updated in place (rows P + N + i); returns out [w][Hq*D]."""
    q, k, v = _c(q, np.uint16), _c(k, np.uint16), _c(v, np.uint16)
    cp = _c(cache_parent, np.int32) if len(cache_parent) else np.zeros(1, np.int32)
    lp = _c(leaf_parent, np.int32)
    w = q.shape[0]
    assert len(lp) == w and k_cache.flags["C_CONTIGUOUS"] and v_cache.flags["C_CONTIGUOUS"]
    S_max = k_cache.shape[1]
    if softmax_scale is None:
        softmax_scale = 1.0 / np.sqrt(D)
    out = np.empty((w, Hq * D), np.uint16)
    rc = _load().oracle_draft_tree_attention(_p(q), q.shape[1], _p(k), _p(v), k.shape[1], _p(k_cache), _p(v_cache),
                                             S_max, P, _p(cp), len(cache_parent), _p(lp), w, Hq, Hkv, D, rope_theta,
                                             softmax_scale, _p(out), Hq * D)
    if rc != 0:
        raise ValueError("oracle_draft_tree_attention: invalid arguments or forest")
    return out


def kv_commit(k_cache, v_cache, P, parent, accepted, n_layers=1, layer_stride=None):
    """In-place commit on [n_layers][Hkv][S_max][D] (or [Hkv][S_max][D]) caches; returns L."""
    p = _c(parent, np.int32)
    assert k_cache.flags["C_CONTIGUOUS"] and v_cache.flags["C_CONTIGUOUS"]
    Hkv, S_max, D = k_cache.shape[-3:]
    if layer_stride is None:
        layer_stride = Hkv * S_max * D
    L = _load().oracle_kv_commit(_p(k_cache), _p(v_cache), n_layers, layer_stride, Hkv, S_max, D,
                                 P, _p(p), len(p), int(accepted))
    if L < 0:
        raise ValueError("oracle_kv_commit: invalid arguments or tree")
    return int(L)


def _w4(W):
    return W4(_p(W["qweight"]), _p(W["scales"]), _p(W["zeros"]))


def verify_layer(dims: dict, weights: dict, k_cache, v_cache, hidden, P, parent):
    """One decoder layer over the tree; returns the new hidden [T][H] (caches updated in place)."""
    h = np.array(hidden, dtype=np.uint16, copy=True, order="C")
    p = _c(parent, np.int32)
    d = Dims(dims["H"], dims["Hq"], dims["Hkv"], dims["D"], dims["F"], dims["S_max"],
             dims.get("eps", 1e-5), dims.get("rope_theta", 500000.0))
    an = _c(weights["attn_norm"], np.uint16)
    mn = _c(weights["mlp_norm"], np.uint16)
    rc = _load().oracle_verify_layer(ctypes.byref(d), _p(an), _p(mn), _w4(weights["wqkv"]),
                                     _w4(weights["wo"]), _w4(weights["wgate"]),
                                     _w4(weights["wup"]), _w4(weights["wdown"]), _p(k_cache),
                                     _p(v_cache), _p(h), len(p), P, _p(p))
    if rc != 0:
        raise ValueError("oracle_verify_layer: invalid arguments or tree")
    return h


def lm_head(h, gamma, W, eps=1e-5):
    h = _c(h, np.uint16)
    M, H = h.shape
    W = _c(W, np.uint16)
    V = W.shape[0]
    out = np.empty((M, V), np.uint16)
    rc = _load().oracle_lm_head(_p(h), M, H, _p(_c(gamma, np.uint16)), eps, _p(W), V, _p(out))
    if rc != 0:
        raise ValueError("oracle_lm_head: invalid arguments")
    return out


def kv_reorganize(k_cache, v_cache, P, parent, last, keep=True, n_layers=1, layer_stride=None):
    """Draft-side reorganisation in place on [n_layers][Hkv][S_max][D] (or
    [Hkv][S_max][D]) caches; returns (L, new_parent of the kept nodes)."""
    p = _c(parent, np.int32)
    assert k_cache.flags["C_CONTIGUOUS"] and v_cache.flags["C_CONTIGUOUS"]
    Hkv, S_max, D = k_cache.shape[-3:]
    if layer_stride is None:
        layer_stride = Hkv * S_max * D
    N = len(p)
    newp = np.empty(max(N, 1), np.int32)
    S = np.zeros(1, np.int32)
    L = _load().oracle_kv_reorganize(_p(k_cache), _p(v_cache), n_layers, layer_stride, Hkv, S_max, D, P,
                                     _p(p if N else np.zeros(1, np.int32)), N, int(last), int(bool(keep)),
                                     _p(newp), _p(S))
    if L < 0:
        raise ValueError("oracle_kv_reorganize: invalid arguments or forest")
    return int(L), newp[:int(S[0])].copy()


def greedy_accept(logits, tokens, parent):
    """Greedy acceptance of a verified tree: (argmax[T], accepted node, bonus
    token, accepted path length L)."""
    lg = _c(logits, np.uint16)
    T, V = lg.shape
    tok = _c(tokens, np.int32)
    p = _c(parent, np.int32)
    assert len(tok) == T and len(p) == T
    am = np.empty(T, np.int32)
    acc = np.zeros(1, np.int32)
    bon = np.zeros(1, np.int32)
    L = _load().oracle_greedy_accept(_p(lg), T, V, V, _p(tok), _p(p), _p(am), _p(acc), _p(bon))
    if L < 0:
        raise ValueError("oracle_greedy_accept: invalid arguments or tree")
    return am, int(acc[0]), int(bon[0]), int(L)


def topk_logprobs(logits, k):
    """The k most probable next tokens of each logits row (ties: lower index
    first) and their log-softmax values: (tokens [n][k] int32, logprobs
    [n][k] float64)."""
    lg = _c(logits, np.uint16)
    n, V = lg.shape
    tok = np.zeros((n, k), np.int32)
    lp = np.zeros((n, k), np.float64)
    assert _load().oracle_topk_logprobs(_p(lg), n, V, V, k, _p(tok), _p(lp)) == 0
    return tok, lp


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the checker's later parallel loops (timing only; every
    result is independent of the thread count)."""
    _load().oracle_set_num_threads(int(n))
