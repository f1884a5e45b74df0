"""Python binding of libswiftspec.so: the tree-verification step of
speculative decoding on AMD Instinct MI355X (gfx950).

Argument marshalling only: every computation runs in the library's HIP
kernels.  PyTorch supplies device memory and the current HIP stream; the
functions below pass tensor pointers, shapes and the stream handle through
the C ABI declared in ``include/swiftspec.h`` and raise ``SwiftSpecError``
on a non-zero status.  There is no fallback: if the compiled library is
missing, importing a function raises.

fp16 tensors may be ``torch.float16`` or ``torch.int16``/``torch.uint16``
views of the same bits.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_build", "libswiftspec.so")

_lib = None

i32, i64, f32, f64, vp, sz = (ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double,
                              ctypes.c_void_p, ctypes.c_size_t)

OK, INVALID_ARG, UNSUPPORTED, MISALIGNED, WORKSPACE_TOO_SMALL, BAD_TREE, HIP_ERROR, CAPACITY = range(8)
DEVERR_BAD_TREE, DEVERR_BAD_PREFIX, DEVERR_BAD_ACCEPTED = 1, 2, 4
WS_HEADER_BYTES = 65536
MAX_TREE = 64
MAX_M = 64


class SwiftSpecError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = _load().swiftspec_status_string(status).decode()
        if status == HIP_ERROR:
            msg += f" (hipError {_load().swiftspec_last_hip_error()})"
        super().__init__(f"{where}: {msg} [status {status}]")
        self.status = status


class W4(ctypes.Structure):
    _fields_ = [("qweight", vp), ("scales", vp), ("zeros", vp), ("K", i32), ("N", i32), ("packed", vp)]


class Dims(ctypes.Structure):
    _fields_ = [("H", i32), ("Hq", i32), ("Hkv", i32), ("D", i32), ("F", i32), ("S_max", i32),
                ("eps", f32), ("rope_theta", f32)]


class Layer(ctypes.Structure):
    _fields_ = [("attn_norm", vp), ("mlp_norm", vp), ("wqkv", W4), ("wo", W4), ("wgate", W4),
                ("wup", W4), ("wdown", W4), ("k_cache", vp), ("v_cache", vp)]


_SIGS = {
    "swiftspec_status_string": ([ctypes.c_int], ctypes.c_char_p),
    "swiftspec_last_hip_error": ([], ctypes.c_int),
    "swiftspec_workspace_init": ([vp, sz, vp], ctypes.c_int),
    "swiftspec_draft_tree_attention": ([vp, i32, vp, vp, i32, vp, vp, i32, vp, vp, i32, vp, i32, i32, i32, i32, vp,
                                        f32, vp, i32, vp, sz, vp], ctypes.c_int),
    "swiftspec_kv_reorganize": ([vp, vp, i32, i64, i32, i32, i32, vp, vp, i32, vp, vp, vp, vp, i32, vp, sz, vp],
                                ctypes.c_int),
    "swiftspec_topk_logprobs_workspace_bytes": ([i32], sz),
    "swiftspec_topk_logprobs": ([vp, i32, i32, i32, i32, vp, vp, vp, sz, vp], ctypes.c_int),
    "swiftspec_draft_tree_create": ([i32, i32, ctypes.POINTER(vp)], ctypes.c_int),
    "swiftspec_draft_tree_destroy": ([vp], None),
    "swiftspec_draft_tree_size": ([vp], i32),
    "swiftspec_draft_tree_rows": ([vp], i32),
    "swiftspec_draft_tree_nodes": ([vp, vp, vp, vp, vp, vp], ctypes.c_int),
    "swiftspec_draft_tree_forest": ([vp, vp], ctypes.c_int),
    "swiftspec_draft_tree_select_leaves": ([vp, i32, vp, vp, vp], ctypes.c_int),
    "swiftspec_draft_tree_expand": ([vp, i32, vp, i32, vp, vp], ctypes.c_int),
    "swiftspec_draft_tree_select_subgraph": ([vp, i32, vp, vp, vp, vp], ctypes.c_int),
    "swiftspec_draft_tree_reroot": ([vp, vp, i32, vp, vp, vp, vp, vp], ctypes.c_int),
    "swiftspec_greedy_accept_workspace_bytes": ([i32], sz),
    "swiftspec_greedy_accept": ([vp, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp], ctypes.c_int),
    "swiftspec_read_device_error": ([vp, vp, ctypes.POINTER(ctypes.c_uint32)], ctypes.c_int),
    "swiftspec_clock_sample": ([vp, i32, vp], ctypes.c_int),
    "swiftspec_w4_packed_bytes": ([i32, i32], sz),
    "swiftspec_w4_prepack": ([ctypes.POINTER(W4), vp, sz, vp], ctypes.c_int),
    "swiftspec_w4a16_gemm": ([ctypes.POINTER(W4), vp, i32, i32, vp, i32, vp, i32, vp, sz, vp], ctypes.c_int),
    "swiftspec_w4a16_gemm_workspace_bytes": ([i32, i32, i32], sz),
    "swiftspec_w4a16_swiglu": ([ctypes.POINTER(W4), ctypes.POINTER(W4), vp, i32, i32, vp, i32, vp, sz, vp],
                               ctypes.c_int),
    "swiftspec_w4a16_swiglu_workspace_bytes": ([i32, i32, i32], sz),
    "swiftspec_prepared_bytes": ([i32, i32], sz),
    "swiftspec_prepare_activations": ([vp, i32, i32, i32, vp, vp], ctypes.c_int),
    "swiftspec_w4a16_gemm_prepared": ([ctypes.POINTER(W4), vp, i32, vp, i32, vp, i32, vp, sz, vp], ctypes.c_int),
    "swiftspec_w4a16_swiglu_prepared": ([ctypes.POINTER(W4), ctypes.POINTER(W4), vp, i32, vp, i32, vp, sz, vp],
                                        ctypes.c_int),
    "swiftspec_rmsnorm": ([vp, i32, i32, i32, vp, f32, vp, i32, vp], ctypes.c_int),
    "swiftspec_rmsnorm_w4a16_gemm": ([ctypes.POINTER(W4), vp, i32, i32, vp, f32, vp, i32, vp, sz, vp],
                                     ctypes.c_int),
    "swiftspec_rmsnorm_w4a16_swiglu": ([ctypes.POINTER(W4), ctypes.POINTER(W4), vp, i32, i32, vp, f32, vp, i32,
                                       vp, sz, vp], ctypes.c_int),
    "swiftspec_tree_attention": ([vp, i32, vp, vp, i32, vp, vp, i32, vp, vp, i32, i32, i32, i32, vp, f32,
                                  vp, i32, vp, sz, vp], ctypes.c_int),
    "swiftspec_tree_attention_workspace_bytes": ([i32, i32, i32, i32, i32], sz),
    "swiftspec_tree_attention_noalloc": ([vp, i32, vp, vp, i32, vp, vp, i32, vp, vp, i32, i32, i32, i32, vp, f32,
                                          vp, i32, vp, vp], ctypes.c_int),
    "swiftspec_rope_table": ([f64, i32, i32, vp], ctypes.c_int),
    "swiftspec_tree_masks": ([vp, i32, i32, vp, vp, vp, vp], ctypes.c_int),
    "swiftspec_tree_validate": ([vp, i32, vp], ctypes.c_int),
    "swiftspec_kv_commit": ([vp, vp, i32, i64, i32, i32, i32, vp, vp, i32, vp, i32, vp, sz, vp], ctypes.c_int),
    "swiftspec_verify_layer": ([ctypes.POINTER(Layer), ctypes.POINTER(Dims), vp, i32, vp, vp, vp, vp, sz, vp],
                               ctypes.c_int),
    "swiftspec_verify_layer_workspace_bytes": ([ctypes.POINTER(Dims), i32], sz),
    "swiftspec_verify_layer_workspace_layout": ([ctypes.POINTER(Dims), i32, ctypes.POINTER(sz)], ctypes.c_int),
    "swiftspec_lm_head": ([vp, i32, i32, vp, f32, vp, i32, vp, vp, sz, vp], ctypes.c_int),
    "swiftspec_lm_head_workspace_bytes": ([i32, i32, i32], sz),
    "swiftspec_verify_step": ([ctypes.POINTER(Layer), i32, ctypes.POINTER(Dims), vp, i32, vp, vp, vp, vp, vp,
                               i32, vp, vp, sz, vp], ctypes.c_int),
    "swiftspec_verify_step_workspace_bytes": ([ctypes.POINTER(Dims), i32, i32], sz),
    "swiftspec_w4a16_gemm_valu": ([ctypes.POINTER(W4), vp, i32, i32, vp, i32, vp, i32, vp, sz, vp], ctypes.c_int),
    "swiftspec_w4a16_gemm_valu_workspace_bytes": ([i32, i32, i32], sz),
    "swiftspec_graph_begin": ([vp], ctypes.c_int),
    "swiftspec_graph_end": ([vp, ctypes.POINTER(vp)], ctypes.c_int),
    "swiftspec_graph_launch": ([vp, vp], ctypes.c_int),
    "swiftspec_graph_destroy": ([vp], ctypes.c_int),
}
EXPORTS = tuple(_SIGS)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"libswiftspec.so is not built ({LIB_PATH}); run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    for name, (args, res) in _SIGS.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def lib():
    return _load()


def _check(status: int, where: str):
    if status != OK:
        raise SwiftSpecError(status, where)


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


# ------------------------------------------------------------------ helpers

def workspace(nbytes: int, device="cuda"):
    """A zero-filled device workspace (its header counters start at zero)."""
    import torch
    return torch.zeros(int(nbytes), dtype=torch.uint8, device=device)


def make_w4(qweight, scales, zeros, packed=None) -> W4:
    """Describe an int4 matrix held in device tensors qweight [N][K/2] u8,
    scales [N][K/128] fp16, zeros [N][K/128] u8, and optionally its
    kernel-native copy `packed` (see prepack_w4)."""
    N, half_k = qweight.shape
    return W4(qweight.data_ptr(), scales.data_ptr(), zeros.data_ptr(), 2 * half_k, N,
              packed.data_ptr() if packed is not None else None)


def packed_bytes(K: int, N: int) -> int:
    return int(_load().swiftspec_w4_packed_bytes(K, N))


def prepack_w4(W: W4, stream=None):
    """Allocate and fill the kernel-native copy of W; returns the uint8
    device tensor and sets W.packed to it (keep the tensor alive)."""
    import torch
    t = torch.empty(packed_bytes(W.K, W.N), dtype=torch.uint8, device="cuda")
    _check(_load().swiftspec_w4_prepack(ctypes.byref(W), _ptr(t), t.numel(), _stream(stream)), "w4_prepack")
    W.packed = t.data_ptr()
    return t


def prepack_w4_into(W: W4, out, stream=None):
    """Fill the caller's uint8 device tensor `out` (at least
    packed_bytes(K, N) bytes, 16-byte aligned) with the kernel-native copy of
    W and set W.packed to it."""
    _check(_load().swiftspec_w4_prepack(ctypes.byref(W), _ptr(out), out.numel(), _stream(stream)), "w4_prepack")
    W.packed = out.data_ptr()


def rope_table(theta: float, S_max: int, D: int):
    """Host fp32 (cos, sin) table [S_max][D/2][2] built in fp64 by the library."""
    import numpy as np
    out = np.empty((S_max, D // 2, 2), np.float32)
    _check(_load().swiftspec_rope_table(theta, S_max, D, out.ctypes.data), "rope_table")
    return out


def tree_validate(parent):
    import numpy as np
    p = np.ascontiguousarray(parent, dtype=np.int32)
    depth = np.empty(len(p), np.int32)
    st = _load().swiftspec_tree_validate(p.ctypes.data, len(p), depth.ctypes.data)
    return st, depth


def read_device_error(ws, stream=None) -> int:
    out = ctypes.c_uint32(0)
    _check(_load().swiftspec_read_device_error(_ptr(ws), _stream(stream), ctypes.byref(out)),
           "read_device_error")
    return int(out.value)


def clock_sample(out, window_us: int = 20, stream=None):
    """Enqueue the clock sample on `stream` into `out` (an int64 device
    tensor of at least 4 elements): shader-clock and real-time counters
    before and after a window_us wait."""
    assert out.numel() >= 4 and out.element_size() == 8
    _check(_load().swiftspec_clock_sample(_ptr(out), window_us, _stream(stream)), "clock_sample")


def clock_ghz(sample) -> float:
    """Shader clock in GHz from a clock_sample result (host sequence of 4)."""
    c0, r0, c1, r1 = (int(v) for v in sample[:4])
    return (c1 - c0) / max(1, r1 - r0) / 10.0


def workspace_init(ws, stream=None):
    _check(_load().swiftspec_workspace_init(_ptr(ws), ws.numel(), _stream(stream)), "workspace_init")


# ------------------------------------------------------------ operations

def gemm_workspace_bytes(M: int, K: int, N: int) -> int:
    return int(_load().swiftspec_w4a16_gemm_workspace_bytes(M, K, N))


def gemm_valu_workspace_bytes(M: int, K: int, N: int) -> int:
    return int(_load().swiftspec_w4a16_gemm_valu_workspace_bytes(M, K, N))


def w4a16_gemm_valu(W: W4, x, y, ws, residual=None, stream=None):
    """As w4a16_gemm, on the vector ALUs only (comparison variant)."""
    st = _load().swiftspec_w4a16_gemm_valu(ctypes.byref(W), _ptr(x), x.shape[0], x.stride(0), _ptr(y), y.stride(0),
                                           _ptr(residual), residual.stride(0) if residual is not None else 0,
                                           _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "w4a16_gemm_valu")


def swiglu_workspace_bytes(M: int, K: int, N: int) -> int:
    return int(_load().swiftspec_w4a16_swiglu_workspace_bytes(M, K, N))


def w4a16_gemm(W: W4, x, y, ws, residual=None, stream=None):
    M, ldx = x.shape[0], x.stride(0)
    st = _load().swiftspec_w4a16_gemm(ctypes.byref(W), _ptr(x), M, ldx, _ptr(y), y.stride(0),
                                      _ptr(residual), residual.stride(0) if residual is not None else 0,
                                      _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "w4a16_gemm")


def w4a16_swiglu(Wg: W4, Wu: W4, x, y, ws, stream=None):
    st = _load().swiftspec_w4a16_swiglu(ctypes.byref(Wg), ctypes.byref(Wu), _ptr(x), x.shape[0],
                                        x.stride(0), _ptr(y), y.stride(0), _ptr(ws), ws.numel(),
                                        _stream(stream))
    _check(st, "w4a16_swiglu")


def prepared_bytes(M: int, K: int) -> int:
    return int(_load().swiftspec_prepared_bytes(M, K))


def prepare_activations(x, xp, stream=None):
    """x [M][>=K] fp16 -> xp (uint8/int16 device buffer of prepared_bytes(M, K))."""
    M, K = x.shape
    _check(_load().swiftspec_prepare_activations(_ptr(x), M, x.stride(0), K, _ptr(xp), _stream(stream)),
           "prepare_activations")


def w4a16_gemm_prepared(W: W4, xp, M: int, y, ws, residual=None, stream=None):
    st = _load().swiftspec_w4a16_gemm_prepared(ctypes.byref(W), _ptr(xp), M, _ptr(y), y.stride(0),
                                               _ptr(residual), residual.stride(0) if residual is not None else 0,
                                               _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "w4a16_gemm_prepared")


def w4a16_swiglu_prepared(Wg: W4, Wu: W4, xp, M: int, y, ws, stream=None):
    st = _load().swiftspec_w4a16_swiglu_prepared(ctypes.byref(Wg), ctypes.byref(Wu), _ptr(xp), M, _ptr(y),
                                                 y.stride(0), _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "w4a16_swiglu_prepared")


def rmsnorm(x, gamma, out, eps=1e-5, stream=None):
    st = _load().swiftspec_rmsnorm(_ptr(x), x.shape[0], x.shape[1], x.stride(0), _ptr(gamma), eps,
                                   _ptr(out), out.stride(0), _stream(stream))
    _check(st, "rmsnorm")


def rmsnorm_w4a16_gemm(W: W4, x, gamma, y, ws, eps=1e-5, stream=None):
    """y = rmsnorm(x, gamma) . W'^T (workspace of gemm_workspace_bytes)."""
    st = _load().swiftspec_rmsnorm_w4a16_gemm(ctypes.byref(W), _ptr(x), x.shape[0], x.stride(0), _ptr(gamma), eps,
                                              _ptr(y), y.stride(0), _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "rmsnorm_w4a16_gemm")


def rmsnorm_w4a16_swiglu(Wg: W4, Wu: W4, x, gamma, y, ws, eps=1e-5, stream=None):
    """y = silu(xn . Wg'^T) * (xn . Wu'^T), xn = rmsnorm(x, gamma)
    (workspace of swiglu_workspace_bytes)."""
    st = _load().swiftspec_rmsnorm_w4a16_swiglu(ctypes.byref(Wg), ctypes.byref(Wu), _ptr(x), x.shape[0],
                                                x.stride(0), _ptr(gamma), eps, _ptr(y), y.stride(0), _ptr(ws),
                                                ws.numel(), _stream(stream))
    _check(st, "rmsnorm_w4a16_swiglu")


def tree_attention_workspace_bytes(T, Hq, Hkv, D, S_max) -> int:
    return int(_load().swiftspec_tree_attention_workspace_bytes(T, Hq, Hkv, D, S_max))


def tree_attention(q, k, v, k_cache, v_cache, prefix_len, parent, Hq, Hkv, D, rope, out, ws,
                   softmax_scale=None, stream=None):
    """q [T][>=Hq*D], k/v [T][>=Hkv*D] (row strides are the leading dims),
    caches [Hkv][S_max][D], prefix_len int32[1] and parent int32[T] on device."""
    T = parent.shape[0]
    S_max = k_cache.shape[-2]
    if softmax_scale is None:
        softmax_scale = 1.0 / (D ** 0.5)
    st = _load().swiftspec_tree_attention(_ptr(q), q.stride(0), _ptr(k), _ptr(v), k.stride(0),
                                          _ptr(k_cache), _ptr(v_cache), S_max, _ptr(prefix_len),
                                          _ptr(parent), T, Hq, Hkv, D, _ptr(rope), softmax_scale,
                                          _ptr(out), out.stride(0), _ptr(ws), ws.numel(),
                                          _stream(stream))
    _check(st, "tree_attention")


NOALLOC_SCRATCH_BYTES = 32 << 20


def tree_attention_noalloc(q, k, v, k_cache, v_cache, prefix_len, parent, Hq, Hkv, D, rope, out, error=None,
                           softmax_scale=None, stream=None):
    """tree_attention without a workspace (partials in the library's own
    device array); error: device int32[1] that receives the device error
    bits, or None."""
    T = parent.shape[0]
    S_max = k_cache.shape[-2]
    if softmax_scale is None:
        softmax_scale = 1.0 / (D ** 0.5)
    st = _load().swiftspec_tree_attention_noalloc(_ptr(q), q.stride(0), _ptr(k), _ptr(v), k.stride(0),
                                                  _ptr(k_cache), _ptr(v_cache), S_max, _ptr(prefix_len),
                                                  _ptr(parent), T, Hq, Hkv, D, _ptr(rope), softmax_scale,
                                                  _ptr(out), out.stride(0), _ptr(error), _stream(stream))
    _check(st, "tree_attention_noalloc")


def tree_masks(parents, anc, depth, status, stream=None):
    n, T = parents.shape
    st = _load().swiftspec_tree_masks(_ptr(parents), n, T, _ptr(anc), _ptr(depth), _ptr(status),
                                      _stream(stream))
    _check(st, "tree_masks")


def kv_commit(k_cache, v_cache, prefix_len, parent, accepted, n_layers=1, layer_stride=None,
              advance=False, ws=None, stream=None):
    """Caches [n_layers][Hkv][S_max][D] (or [Hkv][S_max][D]); prefix_len,
    parent and accepted are device int32 tensors."""
    Hkv, S_max, D = k_cache.shape[-3:]
    if layer_stride is None:
        layer_stride = Hkv * S_max * D
    st = _load().swiftspec_kv_commit(_ptr(k_cache), _ptr(v_cache), n_layers, layer_stride, Hkv, S_max,
                                     D, _ptr(prefix_len), _ptr(parent), parent.shape[0], _ptr(accepted),
                                     int(bool(advance)), _ptr(ws), ws.numel() if ws is not None else 0,
                                     _stream(stream))
    _check(st, "kv_commit")


def draft_tree_attention(q, k, v, k_cache, v_cache, prefix_len, cache_parent, leaf_parent, Hq, Hkv, rope, out, ws,
                         softmax_scale=None, stream=None):
    """Draft-model attention with the non-square mask: q [w][>=Hq*D],
    k / v [w][>=Hkv*D] (strided views allowed), caches [Hkv][S_max][D],
    cache_parent [N] (None or empty for N = 0) and leaf_parent [w] device
    int32."""
    Hkv_, S_max, D = k_cache.shape
    w = q.shape[0]
    N = 0 if cache_parent is None else cache_parent.shape[0]
    scale = softmax_scale if softmax_scale is not None else 1.0 / (D ** 0.5)
    st = _load().swiftspec_draft_tree_attention(_ptr(q), q.stride(0), _ptr(k), _ptr(v), k.stride(0), _ptr(k_cache),
                                                _ptr(v_cache), S_max, _ptr(prefix_len),
                                                _ptr(cache_parent) if N else None, N, _ptr(leaf_parent), w, Hq, Hkv,
                                                D, _ptr(rope), scale, _ptr(out), out.stride(0), _ptr(ws), ws.numel(),
                                                _stream(stream))
    _check(st, "draft_tree_attention")


def kv_reorganize(k_cache, v_cache, prefix_len, parent, last, keep, new_parent=None, n_kept=None, n_layers=1,
                  layer_stride=None, advance=False, ws=None, stream=None):
    """Draft-side reorganisation on caches [n_layers][Hkv][S_max][D] (or
    [Hkv][S_max][D]); prefix_len, parent [N], last, keep and the outputs
    new_parent [N], n_kept are device int32 tensors."""
    Hkv, S_max, D = k_cache.shape[-3:]
    if layer_stride is None:
        layer_stride = Hkv * S_max * D
    st = _load().swiftspec_kv_reorganize(_ptr(k_cache), _ptr(v_cache), n_layers, layer_stride, Hkv, S_max, D,
                                         _ptr(prefix_len), _ptr(parent), parent.shape[0], _ptr(last), _ptr(keep),
                                         _ptr(new_parent), _ptr(n_kept), int(bool(advance)), _ptr(ws),
                                         ws.numel() if ws is not None else 0, _stream(stream))
    _check(st, "kv_reorganize")


def greedy_accept_workspace_bytes(T) -> int:
    return int(_load().swiftspec_greedy_accept_workspace_bytes(T))


def greedy_accept(logits, tokens, parent, argmax, accepted, bonus, ws, path_len=None, V=None,
                  stream=None):
    """logits [T][ldl] fp16 (first V columns; default all); tokens, parent
    [T] and the outputs argmax [T], accepted, bonus, path_len [1] are device
    int32 tensors."""
    T, ldl = logits.shape
    st = _load().swiftspec_greedy_accept(_ptr(logits), ldl, T, ldl if V is None else V, _ptr(tokens),
                                         _ptr(parent), _ptr(argmax), _ptr(accepted), _ptr(bonus),
                                         _ptr(path_len), _ptr(ws), ws.numel() if ws is not None else 0,
                                         _stream(stream))
    _check(st, "greedy_accept")


def topk_logprobs_workspace_bytes(n) -> int:
    return int(_load().swiftspec_topk_logprobs_workspace_bytes(n))


def topk_logprobs(logits, tokens, logprobs, ws, V=None, stream=None):
    """logits [n][ldl] fp16 (first V columns; default all) -> the k most
    probable tokens of each row (device int32 tokens [n][k]) and their
    log-softmax values (device float32 logprobs [n][k])."""
    n, ldl = logits.shape
    k = tokens.shape[1]
    st = _load().swiftspec_topk_logprobs(_ptr(logits), ldl, n, ldl if V is None else V, k, _ptr(tokens),
                                         _ptr(logprobs), _ptr(ws), ws.numel() if ws is not None else 0,
                                         _stream(stream))
    _check(st, "topk_logprobs")


class DraftTree:
    """Host-side draft tree (swiftspec_draft_tree_*): host numpy arrays in
    and out, no device work."""

    def __init__(self, capacity: int, root_token: int):
        import numpy as np
        self._np = np
        h = vp()
        _check(_load().swiftspec_draft_tree_create(capacity, root_token, ctypes.byref(h)), "draft_tree_create")
        self._h = h

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.swiftspec_draft_tree_destroy(self._h)
            self._h = None

    def _a(self, n, dtype):
        return self._np.zeros(max(int(n), 1), dtype)

    @staticmethod
    def _p(a):
        return a.ctypes.data if a is not None else None

    def size(self) -> int:
        return int(_load().swiftspec_draft_tree_size(self._h))

    def rows(self) -> int:
        return int(_load().swiftspec_draft_tree_rows(self._h))

    def nodes(self):
        """(token, parent, weight, row, expanded) arrays over all nodes."""
        np = self._np
        n = self.size()
        tok, par, row, exp = (self._a(n, np.int32) for _ in range(4))
        w = self._a(n, np.float64)
        _check(_load().swiftspec_draft_tree_nodes(self._h, self._p(tok), self._p(par), self._p(w), self._p(row),
                                                  self._p(exp)), "draft_tree_nodes")
        return tok[:n], par[:n], w[:n], row[:n], exp[:n]

    def forest(self):
        f = self._a(self.rows(), self._np.int32)
        _check(_load().swiftspec_draft_tree_forest(self._h, self._p(f)), "draft_tree_forest")
        return f[:self.rows()]

    def select_leaves(self, w: int):
        np = self._np
        leaves, prow, n = self._a(w, np.int32), self._a(w, np.int32), np.zeros(1, np.int32)
        _check(_load().swiftspec_draft_tree_select_leaves(self._h, w, self._p(leaves), self._p(prow),
                                                          self._p(n)), "draft_tree_select_leaves")
        return leaves[:n[0]], prow[:n[0]]

    def expand(self, leaves, tokens, logprobs):
        np = self._np
        leaves = np.ascontiguousarray(leaves, np.int32)
        tokens = np.ascontiguousarray(tokens, np.int32).reshape(len(leaves), -1)
        logprobs = np.ascontiguousarray(logprobs, np.float32).reshape(len(leaves), -1)
        _check(_load().swiftspec_draft_tree_expand(self._h, len(leaves), self._p(leaves), tokens.shape[1],
                                                   self._p(tokens), self._p(logprobs)), "draft_tree_expand")

    def select_subgraph(self, bs: int):
        """(nodes, parent positions, tokens) of the bs most probable nodes."""
        np = self._np
        nodes, par, tok, n = self._a(bs, np.int32), self._a(bs, np.int32), self._a(bs, np.int32), np.zeros(1, np.int32)
        _check(_load().swiftspec_draft_tree_select_subgraph(self._h, bs, self._p(nodes), self._p(par), self._p(tok),
                                                            self._p(n)), "draft_tree_select_subgraph")
        m = int(n[0])
        return nodes[:m], par[:m], tok[:m]

    def reroot(self, verified):
        """dict(last, path_rows, keep, pending) as swiftspec_draft_tree_reroot."""
        np = self._np
        ver = np.ascontiguousarray(verified, np.int32)
        out = np.zeros(4, np.int32)
        pend = self._a(len(ver), np.int32)
        _check(_load().swiftspec_draft_tree_reroot(self._h, self._p(ver), len(ver), self._p(out[0:1]),
                                                   self._p(out[1:2]), self._p(out[2:3]), self._p(pend),
                                                   self._p(out[3:4])), "draft_tree_reroot")
        return {"last": int(out[0]), "path_rows": int(out[1]), "keep": int(out[2]),
                "pending": [int(x) for x in pend[:out[3]]]}


def make_dims(H, Hq, Hkv, D, F, S_max, eps=1e-5, rope_theta=500000.0) -> Dims:
    return Dims(H, Hq, Hkv, D, F, S_max, eps, rope_theta)


def make_layer(attn_norm, mlp_norm, wqkv: W4, wo: W4, wgate: W4, wup: W4, wdown: W4, k_cache,
               v_cache) -> Layer:
    return Layer(attn_norm.data_ptr(), mlp_norm.data_ptr(), wqkv, wo, wgate, wup, wdown,
                 k_cache.data_ptr(), v_cache.data_ptr())


def verify_layer_workspace_bytes(dims: Dims, T: int) -> int:
    return int(_load().swiftspec_verify_layer_workspace_bytes(ctypes.byref(dims), T))


def verify_layer_intermediates(dims: Dims, T: int, ws):
    """Views (int16 bits) of the layer intermediates qkv, o, h, m held in a
    verify_layer workspace."""
    offs = (sz * 4)()
    _check(_load().swiftspec_verify_layer_workspace_layout(ctypes.byref(dims), T, offs),
           "verify_layer_workspace_layout")
    import torch
    n_qkv = (dims.Hq + 2 * dims.Hkv) * dims.D
    cols = [n_qkv, dims.Hq * dims.D, dims.H, dims.F]
    names = ["qkv", "o", "h", "m"]
    out = {}
    for name, off, c in zip(names, offs, cols):
        out[name] = ws[off:off + T * c * 2].view(torch.int16).view(T, c)
    return out


def verify_layer(layer: Layer, dims: Dims, hidden, prefix_len, parent, rope, ws, stream=None):
    st = _load().swiftspec_verify_layer(ctypes.byref(layer), ctypes.byref(dims), _ptr(hidden),
                                        hidden.shape[0], _ptr(prefix_len), _ptr(parent), _ptr(rope),
                                        _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "verify_layer")


def lm_head_workspace_bytes(M, H, V) -> int:
    return int(_load().swiftspec_lm_head_workspace_bytes(M, H, V))


def lm_head(h, gamma, W, logits, ws, eps=1e-5, stream=None):
    M, H = h.shape
    V = W.shape[0]
    st = _load().swiftspec_lm_head(_ptr(h), M, H, _ptr(gamma), eps, _ptr(W), V, _ptr(logits), _ptr(ws),
                                   ws.numel(), _stream(stream))
    _check(st, "lm_head")


def verify_step_workspace_bytes(dims: Dims, T: int, V: int) -> int:
    return int(_load().swiftspec_verify_step_workspace_bytes(ctypes.byref(dims), T, V))


def make_layers(layers):
    """A contiguous ctypes array of Layer descriptors for verify_step."""
    arr = (Layer * len(layers))()
    for i, l in enumerate(layers):
        arr[i] = l
    return arr


def verify_step(layers, dims: Dims, hidden, prefix_len, parent, rope, ws, final_norm=None, lm_head_w=None,
                logits=None, stream=None):
    """All decoder layers in order, then (if lm_head_w is given) the final
    RMSNorm and LM head into logits.  `layers` is a make_layers() array."""
    V = 0 if lm_head_w is None else lm_head_w.shape[0]
    st = _load().swiftspec_verify_step(layers, len(layers), ctypes.byref(dims), _ptr(hidden), hidden.shape[0],
                                       _ptr(prefix_len), _ptr(parent), _ptr(rope), _ptr(final_norm),
                                       _ptr(lm_head_w), V, _ptr(logits), _ptr(ws), ws.numel(), _stream(stream))
    _check(st, "verify_step")


class Graph:
    """A HIP graph captured from the library calls issued on `stream`
    between begin() and end()."""

    def __init__(self):
        self._g = ctypes.c_void_p(None)

    def begin(self, stream=None):
        _check(_load().swiftspec_graph_begin(_stream(stream)), "graph_begin")

    def end(self, stream=None):
        _check(_load().swiftspec_graph_end(_stream(stream), ctypes.byref(self._g)), "graph_end")

    def launch(self, stream=None):
        _check(_load().swiftspec_graph_launch(self._g, _stream(stream)), "graph_launch")

    def __del__(self):
        if self._g and self._g.value and _lib is not None:
            _lib.swiftspec_graph_destroy(self._g)
            self._g = ctypes.c_void_p(None)
