"""CPU checks of the C ABI: the library loads, exports every entry point the
header declares, and rejects bad arguments on the host before any launch."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "swiftspec.h")


@pytest.fixture(scope="module")
def ss():
    import paper_2506_11309_amd as ss
    if not os.path.exists(ss.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    ss.lib()
    return ss


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(swiftspec_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(ss):
    names = _declared()
    assert len(names) >= 20
    lib = ctypes.CDLL(ss.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(ss.EXPORTS) == names


def test_status_strings(ss):
    lib = ss.lib()
    for code in range(7):
        assert lib.swiftspec_status_string(code)
    assert lib.swiftspec_status_string(99) == b"unknown status"


def test_host_side_validation_rejects_before_launch(ss):
    lib = ss.lib()
    fake = 0x10000  # never dereferenced: validation fails first
    W = ss.W4(fake, fake, fake, 4096, 1024, fake)
    ws_small = 16
    # null weight descriptor
    assert lib.swiftspec_w4a16_gemm(None, fake, 8, 4096, fake, 1024, None, 0, fake, 1 << 30, None) == ss.INVALID_ARG
    # K not a multiple of the quantisation group
    W_bad = ss.W4(fake, fake, fake, 4000, 1024, fake)
    W_unpacked = ss.W4(fake, fake, fake, 4096, 1024, None)
    assert lib.swiftspec_w4a16_gemm(ctypes.byref(W_unpacked), fake, 8, 4096, fake, 1024, None, 0, fake, 1 << 30,
                                    None) == ss.INVALID_ARG
    assert lib.swiftspec_w4_packed_bytes(4096, 1024) == 4096 * 1024 // 2 + 1024 * 32 * 4
    assert lib.swiftspec_w4a16_gemm(ctypes.byref(W_bad), fake, 8, 4096, fake, 1024, None, 0, fake, 1 << 30,
                                    None) == ss.UNSUPPORTED
    # too many rows
    assert lib.swiftspec_w4a16_gemm(ctypes.byref(W), fake, 65, 4096, fake, 1024, None, 0, fake, 1 << 30,
                                    None) == ss.UNSUPPORTED
    # a kernel-native copy of 4 GiB or more (past the kernels' 32-bit buffer ranges)
    W_huge = ss.W4(fake, fake, fake, 131072, 65536, fake)
    assert lib.swiftspec_w4_packed_bytes(131072, 65536) > 0xFFFFFFFF
    assert lib.swiftspec_w4a16_gemm(ctypes.byref(W_huge), fake, 8, 131072, fake, 65536, None, 0, fake, 1 << 40,
                                    None) == ss.UNSUPPORTED
    W_edge = ss.W4(fake, fake, fake, 65536, 65536, fake)  # 2 GiB + scales: accepted by the shape check
    assert lib.swiftspec_w4_packed_bytes(65536, 65536) < 0xFFFFFFFF
    assert lib.swiftspec_w4a16_gemm(ctypes.byref(W_edge), fake, 8, 65536, fake, 65536, None, 0, fake, 16,
                                    None) == ss.WORKSPACE_TOO_SMALL
    # misaligned activations / leading dimension
    assert lib.swiftspec_w4a16_gemm(ctypes.byref(W), fake + 2, 8, 4096, fake, 1024, None, 0, fake, 1 << 30,
                                    None) == ss.MISALIGNED
    assert lib.swiftspec_w4a16_gemm(ctypes.byref(W), fake, 8, 4100, fake, 1024, None, 0, fake, 1 << 30,
                                    None) == ss.MISALIGNED
    # workspace too small
    assert lib.swiftspec_w4a16_gemm(ctypes.byref(W), fake, 8, 4096, fake, 1024, None, 0, fake, ws_small,
                                    None) == ss.WORKSPACE_TOO_SMALL
    # attention: unsupported head dim, tree too large
    args = lambda T, D: (fake, 4096, fake, fake, 1024, fake, fake, 4096, fake, fake, T, 32, 8, D, fake, 0.1,
                         fake, 4096, fake, 1 << 30, None)
    assert lib.swiftspec_tree_attention(*args(8, 96)) == ss.UNSUPPORTED
    assert lib.swiftspec_tree_attention(*args(65, 128)) == ss.UNSUPPORTED
    # commit: layer stride too small
    assert lib.swiftspec_kv_commit(fake, fake, 2, 100, 8, 64, 128, fake, fake, 8, fake, 0, None, 0,
                                   None) == ss.INVALID_ARG
    assert lib.swiftspec_graph_begin(None) == ss.INVALID_ARG
    # RMSNorm rows: whole 32-element chunks
    assert lib.swiftspec_rmsnorm(fake, 4, 72, 72, fake, ctypes.c_float(1e-5), fake, 72, None) == ss.UNSUPPORTED
    # RMSNorm + projection: null gamma / up matrix, misaligned gamma, short
    # leading dimension, too many rows, mismatched SwiGLU pair, workspace
    eps = ctypes.c_float(1e-5)
    ng = lambda gam=fake, M=8, ldx=4096, wsb=1 << 30: lib.swiftspec_rmsnorm_w4a16_gemm(
        ctypes.byref(W), fake, M, ldx, gam, eps, fake, 1024, fake, wsb, None)
    assert ng(gam=None) == ss.INVALID_ARG
    assert ng(gam=fake + 2) == ss.MISALIGNED
    assert ng(ldx=4088) == ss.INVALID_ARG
    assert ng(M=65) == ss.UNSUPPORTED
    assert ng(wsb=16) == ss.WORKSPACE_TOO_SMALL
    W_other = ss.W4(fake, fake, fake, 4096, 2048, fake)
    assert lib.swiftspec_rmsnorm_w4a16_swiglu(ctypes.byref(W), None, fake, 8, 4096, fake, eps, fake, 1024, fake,
                                              1 << 30, None) == ss.INVALID_ARG
    assert lib.swiftspec_rmsnorm_w4a16_swiglu(ctypes.byref(W), ctypes.byref(W_other), fake, 8, 4096, fake, eps,
                                              fake, 2048, fake, 1 << 30, None) == ss.INVALID_ARG
    assert lib.swiftspec_rmsnorm_w4a16_swiglu(ctypes.byref(W), ctypes.byref(W), fake, 8, 4096, fake, eps, fake,
                                              1024, fake, 16, None) == ss.WORKSPACE_TOO_SMALL
    # greedy acceptance: sizes, leading dimension, workspace, null outputs
    acc = lambda T, V, ldl, lg=fake, ws=fake, wsb=1 << 20, bonus=fake: lib.swiftspec_greedy_accept(
        lg, ldl, T, V, fake, fake, fake, fake, bonus, None, ws, wsb, None)
    assert acc(0, 1000, 1000) == ss.INVALID_ARG
    assert acc(65, 1000, 1000) == ss.UNSUPPORTED
    assert acc(8, 1000, 999) == ss.INVALID_ARG
    assert acc(8, 1000, 1004) == ss.MISALIGNED
    assert acc(8, 1000, 1000, lg=fake + 4) == ss.MISALIGNED
    assert acc(8, 1000, 1000, wsb=16) == ss.WORKSPACE_TOO_SMALL
    assert acc(8, 1000, 1000, ws=None) == ss.INVALID_ARG
    assert acc(8, 1000, 1000, bonus=None) == ss.INVALID_ARG
    assert lib.swiftspec_greedy_accept_workspace_bytes(64) >= ss.WS_HEADER_BYTES + 64 * 16 * 8
    # draft attention: tree-cache size, missing forest, leaf count
    dargs = lambda N, w=8, cp=fake: (fake, 2048, fake, fake, 512, fake, fake, 4096, fake, cp, N, fake, w, 32, 8, 64,
                                     fake, ctypes.c_float(0.125), fake, 2048, fake, 1 << 30, None)
    assert lib.swiftspec_draft_tree_attention(*dargs(65)) == ss.UNSUPPORTED
    assert lib.swiftspec_draft_tree_attention(*dargs(4, cp=None)) == ss.INVALID_ARG
    assert lib.swiftspec_draft_tree_attention(*dargs(4, w=65)) == ss.UNSUPPORTED
    assert lib.swiftspec_draft_tree_attention(*dargs(-1)) == ss.INVALID_ARG
    # draft-side reorganisation: forest size, head dim, layer stride, nulls
    reorg = lambda N, D=128, stride=8 * 200 * 128, last=fake: lib.swiftspec_kv_reorganize(
        fake, fake, 2, stride, 8, 200, D, fake, fake, N, last, fake, None, None, 0, None, 0, None)
    assert reorg(0) == ss.INVALID_ARG
    assert reorg(65) == ss.UNSUPPORTED
    assert reorg(8, D=100) == ss.UNSUPPORTED
    assert reorg(8, stride=100) == ss.INVALID_ARG
    assert reorg(8, last=None) == ss.INVALID_ARG
    # allocation-free attention: partials beyond the library's scratch array
    # (1024 KV heads of 64 tokens: 2048 partials of 16.6 KB) are refused
    na = lambda Hq, Hkv, T=64: lib.swiftspec_tree_attention_noalloc(fake, Hq * 128, fake, fake, Hkv * 128, fake,
                                                                    fake, 4096 + T, fake, fake, T, Hq, Hkv, 128,
                                                                    fake, 0.088, fake, Hq * 128, None, None)
    assert na(1024, 1024) == ss.WORKSPACE_TOO_SMALL
    assert na(64, 8, T=65) == ss.UNSUPPORTED
    assert lib.swiftspec_tree_attention_noalloc(None, 8192, fake, fake, 1024, fake, fake, 4128, fake, fake, 32,
                                                64, 8, 128, fake, 0.088, fake, 8192, None, None) == ss.INVALID_ARG
    # the renumbered forest may not be written over the forest being read
    alias = lambda par, newp: lib.swiftspec_kv_reorganize(fake, fake, 2, 8 * 200 * 128, 8, 200, 128, fake, par, 8,
                                                          fake, fake, newp, None, 0, None, 0, None)
    assert alias(fake, fake) == ss.INVALID_ARG
    assert alias(fake, fake + 16) == ss.INVALID_ARG  # overlaps d_parent[4 .. 8)
    assert alias(fake + 16, fake) == ss.INVALID_ARG
    # draft expansion (top-k log-softmax): rows, k, leading dimension, workspace
    topk = lambda n, V, ldl, k, lg=fake, wsb=1 << 20: lib.swiftspec_topk_logprobs(lg, ldl, n, V, k, fake, fake, fake,
                                                                                   wsb, None)
    assert topk(0, 1000, 1000, 4) == ss.INVALID_ARG
    assert topk(65, 1000, 1000, 4) == ss.UNSUPPORTED
    assert topk(8, 1000, 1000, 9) == ss.UNSUPPORTED
    assert topk(8, 1000, 1000, 0) == ss.INVALID_ARG
    assert topk(8, 4, 8, 5) == ss.INVALID_ARG  # k > V
    assert topk(8, 1000, 1004, 4) == ss.MISALIGNED
    assert topk(8, 1000, 1000, 4, lg=fake + 2) == ss.MISALIGNED
    assert topk(8, 1000, 1000, 4, wsb=16) == ss.WORKSPACE_TOO_SMALL
    assert lib.swiftspec_topk_logprobs_workspace_bytes(8) >= ss.WS_HEADER_BYTES + 8 * 64 * 9 * 8


def test_verify_step_rejects_before_launch(ss):
    lib = ss.lib()
    fake = 0x10000  # never dereferenced: validation fails first
    H, Hq, Hkv, D, F, S = 2048, 32, 8, 64, 8192, 1024
    d = ss.make_dims(H, Hq, Hkv, D, F, S)
    w = lambda K, N: ss.W4(fake, fake, fake, K, N, fake)
    good = ss.Layer(fake, fake, w(H, (Hq + 2 * Hkv) * D), w(Hq * D, H), w(H, F), w(H, F), w(F, H), fake, fake)
    bad = ss.Layer(fake, fake, w(H, (Hq + 2 * Hkv) * D), w(Hq * D, H), w(H, F), w(H, F), w(F, H), None, fake)
    wrong = ss.Layer(fake, fake, w(H, (Hq + 2 * Hkv) * D), w(Hq * D, H), w(H, F), w(H, 2 * F), w(F, H), fake, fake)
    ws = 1 << 40

    def step(layers, n, V, T=8, ws_bytes=ws, logits=fake):
        return lib.swiftspec_verify_step(ss.make_layers(layers), n, ctypes.byref(d), fake, T, fake, fake, fake,
                                         fake, fake, V, logits, fake, ws_bytes, None)

    assert step([good], 0, 0) == ss.INVALID_ARG          # nothing to do
    assert step([good], 1, 24) == ss.UNSUPPORTED         # V % 16 != 0
    assert step([good], 1, 32, logits=None) == ss.INVALID_ARG
    assert step([good, bad], 2, 0) == ss.INVALID_ARG     # a later layer's null cache: nothing enqueued
    assert step([good, wrong], 2, 0) == ss.INVALID_ARG   # a later layer's mismatched shape
    assert step([good], 1, 32, T=65) == ss.UNSUPPORTED
    assert step([good], 1, 32, ws_bytes=16) == ss.WORKSPACE_TOO_SMALL
    step_ws = ss.verify_step_workspace_bytes(d, 8, 32000)
    assert step_ws >= ss.verify_layer_workspace_bytes(d, 8)
    assert step_ws >= lib.swiftspec_lm_head_workspace_bytes(8, H, 32000)


def test_workspace_queries(ss):
    lib = ss.lib()
    for M, K, N in ((8, 2048, 3072), (32, 8192, 10240), (64, 28672, 8192)):
        assert lib.swiftspec_w4a16_gemm_workspace_bytes(M, K, N) >= ss.WS_HEADER_BYTES
        assert lib.swiftspec_w4a16_swiglu_workspace_bytes(M, K, N) >= ss.WS_HEADER_BYTES
    d = ss.make_dims(8192, 64, 8, 128, 28672, 4128)
    assert ss.verify_layer_workspace_bytes(d, 32) > ss.WS_HEADER_BYTES + 32 * (3 * 8192 + 28672) * 2


def test_tree_validate(ss):
    st, depth = ss.tree_validate([-1, 0, 0, 1, 3])
    assert st == ss.OK and depth.tolist() == [0, 1, 1, 2, 3]
    assert ss.tree_validate([-1, 0, 2])[0] == ss.BAD_TREE
    assert ss.tree_validate([0, 0])[0] == ss.BAD_TREE


def test_rope_table_is_fp32_rounding_of_fp64_angles(ss):
    S, D, theta = 300, 128, 500000.0
    t = ss.rope_table(theta, S, D)
    pos = np.arange(S, dtype=np.float64)[:, None]
    inv = theta ** (-2.0 * np.arange(D // 2) / D)
    ang = pos * inv[None, :]
    assert np.array_equal(t[..., 0], np.cos(ang).astype(np.float32))
    assert np.array_equal(t[..., 1], np.sin(ang).astype(np.float32))


def test_clock_sample_rejects_before_launch(ss):
    lib = ss._load()
    assert lib.swiftspec_clock_sample(None, 20, None) == ss.INVALID_ARG
    assert lib.swiftspec_clock_sample(ctypes.c_void_p(8), 0, None) == ss.INVALID_ARG
    assert lib.swiftspec_clock_sample(ctypes.c_void_p(8), 1001, None) == ss.INVALID_ARG
    assert lib.swiftspec_clock_sample(ctypes.c_void_p(12), 20, None) == ss.INVALID_ARG
    assert ss.clock_ghz([1000, 0, 2000, 50]) == 2.0
