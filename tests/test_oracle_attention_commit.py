"""Pins of the fp64 reference checker's tree attention, KV commit and whole
layer, against textbook causal attention, single-token decode, closed forms,
exhaustive small trees and the speculative-decoding equivalence "a tree run
restricted to the accepted path equals a chain run of that path"."""
import itertools

import numpy as np
import pytest

import gen
import oracle


def f64(bits):
    return np.asarray(bits).view(np.float16).astype(np.float64)


def f16bits(x):
    return np.asarray(x, np.float64).astype(np.float16).view(np.uint16)


def _inputs(T, Hq, Hkv, D, P, seed):
    q = gen.normal_f16(seed, 0, (T, Hq * D))
    k = gen.normal_f16(seed, 1, (T, Hkv * D))
    v = gen.normal_f16(seed, 2, (T, Hkv * D))
    kc = np.zeros((Hkv, P + T, D), np.uint16)
    vc = np.zeros((Hkv, P + T, D), np.uint16)
    kc[:, :P] = gen.normal_f16(seed, 3, (Hkv, P, D))
    vc[:, :P] = gen.normal_f16(seed, 4, (Hkv, P, D))
    return q, k, v, kc, vc


def _decode_reference(qvec, pos, keys_rot_f16, vals_f16, D):
    """Textbook single-query softmax attention over the given (already
    rotated, fp16-rounded) keys."""
    qr = oracle.rope(qvec, pos)
    s = (f64(keys_rot_f16) @ qr) / np.sqrt(D)
    p = np.exp(s - s.max())
    return (p @ f64(vals_f16)) / p.sum()


def _assert_close_bits(got, ref):
    d = np.abs(got.astype(np.int32) - ref.astype(np.int32))
    assert d.max() <= 1, d.max()
    assert (d == 0).mean() > 0.98


@pytest.mark.parametrize("T,P,Hq,Hkv,D", [(1, 0, 2, 1, 64), (6, 9, 4, 2, 64), (8, 33, 2, 2, 128)])
def test_chain_tree_equals_causal_attention(T, P, Hq, Hkv, D):
    q, k, v, kc, vc = _inputs(T, Hq, Hkv, D, P, seed=100 + T)
    parent = np.arange(-1, T - 1, dtype=np.int32)
    out = oracle.tree_attention(q, k, v, kc, vc, P, parent, Hq, Hkv, D)
    G = Hq // Hkv
    causal = np.tril(np.ones((T, T), bool))
    ref = np.empty((T, Hq * D))
    for h in range(Hq):
        g = h // G
        # keys of the chain, rotated at positions P + i
        krot = np.stack([f16bits(oracle.rope(f64(k[i, g * D:(g + 1) * D]), P + i)) for i in range(T)])
        for i in range(T):
            keys = np.concatenate([kc[g, :P], krot[causal[i]]])
            vals = np.concatenate([vc[g, :P], v[causal[i], g * D:(g + 1) * D]])
            ref[i, h * D:(h + 1) * D] = _decode_reference(f64(q[i, h * D:(h + 1) * D]), P + i, keys,
                                                          vals, D)
    _assert_close_bits(out, f16bits(ref))
    # cache rows: rotated keys and copied values at rows P + i
    for g in range(Hkv):
        for i in range(T):
            assert np.array_equal(kc[g, P + i], f16bits(oracle.rope(f64(k[i, g * D:(g + 1) * D]), P + i)))
            assert np.array_equal(vc[g, P + i], v[i, g * D:(g + 1) * D])


def test_star_tree_equals_independent_decodes_over_prefix_and_root():
    T, P, Hq, Hkv, D = 7, 20, 2, 1, 64
    q, k, v, kc, vc = _inputs(T, Hq, Hkv, D, P, seed=7)
    parent = np.array([-1] + [0] * (T - 1), np.int32)
    out = oracle.tree_attention(q, k, v, kc, vc, P, parent, Hq, Hkv, D)
    root_k = f16bits(oracle.rope(f64(k[0, :D]), P))
    for i in range(1, T):
        ki = f16bits(oracle.rope(f64(k[i, :D]), P + 1))
        keys = np.concatenate([kc[0, :P], root_k[None], ki[None]])
        vals = np.concatenate([vc[0, :P], v[0:1, :D], v[i:i + 1, :D]])
        for h in range(Hq):
            ref = _decode_reference(f64(q[i, h * D:(h + 1) * D]), P + 1, keys, vals, D)
            _assert_close_bits(out[i, h * D:(h + 1) * D], f16bits(ref))


def test_zero_query_gives_mean_of_visible_values():
    T, P, Hq, Hkv, D = 9, 13, 2, 2, 64
    _, k, v, kc, vc = _inputs(T, Hq, Hkv, D, P, seed=8)
    q = np.zeros((T, Hq * D), np.uint16)
    parent = gen.tree(T, 4, 3, 55)
    depth, anc = oracle.tree(parent)
    out = oracle.tree_attention(q, k, v, kc, vc, P, parent, Hq, Hkv, D)
    for h in range(Hq):
        for i in range(T):
            rows = np.concatenate([vc[h, :P], v[anc[i].astype(bool), h * D:(h + 1) * D]])
            _assert_close_bits(out[i, h * D:(h + 1) * D], f16bits(f64(rows).mean(axis=0)))


def test_non_ancestor_perturbation_leaves_rows_bitwise_unchanged():
    T, P, Hq, Hkv, D = 16, 11, 4, 2, 64
    q, k, v, kc, vc = _inputs(T, Hq, Hkv, D, P, seed=9)
    parent = gen.tree(T, 6, 3, 77)
    depth, anc = oracle.tree(parent)
    base = oracle.tree_attention(q, k, v, kc.copy(), vc.copy(), P, parent, Hq, Hkv, D)
    for i in range(T):
        others = ~anc[i].astype(bool)
        q2, k2, v2 = q.copy(), k.copy(), v.copy()
        noise = gen.normal_f16(1000 + i, 0, q.shape)
        q2[others] = noise[others]
        k2[others] = noise[others][:, :Hkv * D]
        v2[others] = noise[others][:, Hkv * D:2 * Hkv * D]
        out = oracle.tree_attention(q2, k2, v2, kc.copy(), vc.copy(), P, parent, Hq, Hkv, D)
        assert np.array_equal(out[i], base[i])


def test_gqa_head_h_reads_kv_head_h_over_group():
    T, P, Hq, Hkv, D = 5, 7, 6, 3, 64
    q, k, v, kc, vc = _inputs(T, Hq, Hkv, D, P, seed=10)
    parent = gen.tree(T, 3, 2, 5)
    out = oracle.tree_attention(q, k, v, kc.copy(), vc.copy(), P, parent, Hq, Hkv, D)
    G = Hq // Hkv
    for h in range(Hq):
        g = h // G
        single = oracle.tree_attention(np.ascontiguousarray(q[:, h * D:(h + 1) * D]),
                                       np.ascontiguousarray(k[:, g * D:(g + 1) * D]),
                                       np.ascontiguousarray(v[:, g * D:(g + 1) * D]),
                                       np.ascontiguousarray(kc[g:g + 1]), np.ascontiguousarray(vc[g:g + 1]),
                                       P, parent, 1, 1, D)
        assert np.array_equal(out[:, h * D:(h + 1) * D], single)


# ------------------------------------------------------------------ commit


def _path_by_closure(parent, node):
    """Root-to-node path: the node's ancestor-or-self set sorted by index
    (indices increase along any root-to-node path when parent[i] < i)."""
    T = len(parent)
    A = np.eye(T, dtype=np.int64)
    for i in range(1, T):
        A[i, parent[i]] = 1
    R = A.copy()
    for _ in range(T):
        R = ((R @ A) > 0).astype(np.int64)
    return np.nonzero(R[node])[0]


@pytest.mark.parametrize("T", [1, 2, 3, 4, 5, 6])
def test_commit_exhaustive_small_trees_equals_out_of_place_gather(T):
    P, Hkv, D = 3, 2, 4
    base_k = gen.normal_f16(200 + T, 0, (Hkv, P + T + 2, D))
    base_v = gen.normal_f16(200 + T, 1, (Hkv, P + T + 2, D))
    for choice in itertools.product(*[range(i) for i in range(1, T)]):
        parent = np.array((-1,) + choice, np.int32)
        for acc in range(T):
            kc, vc = base_k.copy(), base_v.copy()
            L = oracle.kv_commit(kc, vc, P, parent, acc)
            path = _path_by_closure(parent, acc)
            assert L == len(path)
            for cache, base in ((kc, base_k), (vc, base_v)):
                exp = base.copy()
                exp[:, P:P + L] = base[:, P + path]
                assert np.array_equal(cache, exp)


def test_commit_chain_and_root_are_identity_and_multilayer_stride():
    nl, Hkv, S, D, P, T = 3, 2, 40, 8, 20, 10
    k = gen.normal_f16(300, 0, (nl, Hkv, S, D))
    v = gen.normal_f16(300, 1, (nl, Hkv, S, D))
    chain = np.arange(-1, T - 1, dtype=np.int32)
    for acc in (T - 1, 0):
        kc, vc = k.copy(), v.copy()
        L = oracle.kv_commit(kc, vc, P, chain, acc, n_layers=nl)
        assert L == acc + 1
        assert np.array_equal(kc, k) and np.array_equal(vc, v)
    parent = gen.tree(T, 5, 3, 9)
    acc = gen.accept_leaf(parent, 3)
    kc, vc = k.copy(), v.copy()
    L = oracle.kv_commit(kc, vc, P, parent, acc, n_layers=nl)
    path = _path_by_closure(parent, acc)
    for layer in range(nl):
        exp = k[layer].copy()
        exp[:, P:P + L] = k[layer][:, P + path]
        assert np.array_equal(kc[layer], exp)


def test_commit_rejects_bad_arguments():
    kc = np.zeros((1, 8, 4), np.uint16)
    with pytest.raises(ValueError):
        oracle.kv_commit(kc, kc.copy(), 2, np.array([-1, 0, 5], np.int32), 1)
    with pytest.raises(ValueError):
        oracle.kv_commit(kc, kc.copy(), 2, np.array([-1, 0, 1], np.int32), 3)
    with pytest.raises(ValueError):
        oracle.kv_commit(kc, kc.copy(), 6, np.array([-1, 0, 1], np.int32), 1)


# ------------------------------------------------------------------- layer


def _tiny_layer(seed=0):
    from gen.workloads import LayerShape, WorkloadConfig, make_layer_weights
    shape = LayerShape(H=256, Hq=4, Hkv=2, D=64, F=384)
    cfg = WorkloadConfig(90 + seed, "tiny", shape, P=9, T=12, levels=5, branching=3)
    return cfg, make_layer_weights(cfg)


def test_layer_tree_restricted_to_path_equals_chain_run_of_that_path():
    """Speculative-decoding equivalence: node outputs and committed KV of the
    accepted path do not depend on the rest of the tree (bitwise in fp64)."""
    from gen.workloads import make_kv_prefix, make_tree
    cfg, w = _tiny_layer()
    s = cfg.shape
    dims = {"H": s.H, "Hq": s.Hq, "Hkv": s.Hkv, "D": s.D, "F": s.F, "S_max": cfg.S_max}
    kc, vc = make_kv_prefix(cfg)
    x = gen.normal_f16(cfg.seeds()["activations"], 0, (cfg.T, s.H))
    parent, acc = make_tree(cfg)
    path = _path_by_closure(parent, acc)
    tk, tv = kc.copy(), vc.copy()
    out_tree = oracle.verify_layer(dims, w, tk, tv, x, cfg.P, parent)
    L = oracle.kv_commit(tk, tv, cfg.P, parent, acc)
    ck, cv = kc.copy(), vc.copy()
    chain = np.arange(-1, L - 1, dtype=np.int32)
    out_chain = oracle.verify_layer(dims, w, ck, cv, np.ascontiguousarray(x[path]), cfg.P, chain)
    assert np.array_equal(out_tree[path], out_chain)
    assert np.array_equal(tk[:, :cfg.P + L], ck[:, :cfg.P + L])
    assert np.array_equal(tv[:, :cfg.P + L], cv[:, :cfg.P + L])
    # and the layer output is a residual update of the input (finite, not identical)
    o = f64(out_tree)
    assert np.all(np.isfinite(o)) and not np.array_equal(out_tree, x)


def _diag_w4(N, K, scale, zero=7):
    """int4 weight whose dequantised matrix is scale * I (on min(N, K)), else 0."""
    qint = np.full((N, K), zero, np.uint8)
    d = np.arange(min(N, K))
    qint[d, d] = zero + 1
    q = (qint[:, 0::2] | (qint[:, 1::2] << 4)).astype(np.uint8)
    s = np.full((N, K // 128), np.float16(scale)).view(np.uint16)
    z = np.full((N, K // 128), zero, np.uint8)
    return {"qweight": q, "scales": s, "zeros": z, "K": K, "N": N}


def _zero_w4(N, K):
    return _diag_w4(N, K, 1.0) | {"qweight": np.full((N, K // 2), 0x77, np.uint8)}


def test_layer_wiring_attention_block_closed_form():
    """Wq = 0, Wk = 0, Wv = I, Wo = I, MLP gate = 0, T = 1, P = 0: the single
    token attends only to itself, so out = fp16(x + rmsnorm(x))."""
    H, Hq, Hkv, D, F = 256, 4, 2, 64, 384
    dims = {"H": H, "Hq": Hq, "Hkv": Hkv, "D": D, "F": F, "S_max": 1}
    Nqkv = (Hq + 2 * Hkv) * D
    wqkv = _zero_w4(Nqkv, H)
    # V rows of Wqkv (output columns [(Hq+Hkv)D, Nqkv)) map hidden[0:Hkv*D] through
    qint = np.full((Nqkv, H), 7, np.uint8)
    for j in range(Hkv * D):
        qint[(Hq + Hkv) * D + j, j] = 8
    wqkv["qweight"] = (qint[:, 0::2] | (qint[:, 1::2] << 4)).astype(np.uint8)
    # attention output head h = v of kv head h // 2; Wo selects head 0 and 2's blocks
    wo = _diag_w4(H, Hq * D, 1.0)
    w = {"attn_norm": gen.normal_f16(1, 0, (H,), 1.0, 0.02), "mlp_norm": gen.normal_f16(1, 1, (H,), 1.0, 0.02),
         "wqkv": wqkv, "wo": wo, "wgate": _zero_w4(F, H), "wup": _diag_w4(F, H, 1.0),
         "wdown": _diag_w4(H, F, 1.0)}
    x = gen.normal_f16(2, 0, (1, H))
    kc = np.zeros((Hkv, 1, D), np.uint16)
    vc = np.zeros((Hkv, 1, D), np.uint16)
    out = oracle.verify_layer(dims, w, kc, vc, x, 0, np.array([-1], np.int32))
    xn = oracle.rmsnorm(x, w["attn_norm"])
    # o[h*D + d] = xn[(h//2)*D + d]; Wo = I so h = x + o over H = Hq*D columns
    o = np.concatenate([xn[0, (h // 2) * D:(h // 2 + 1) * D] for h in range(Hq)])
    exp = f16bits(f64(x[0]) + f64(o))
    assert np.array_equal(out[0], exp)


def test_layer_wiring_mlp_block_closed_form():
    """Wo = 0 makes h = x; Wg = I, Wu = 2I, Wd = I give
    out = fp16(x + fp16(silu(hn) * 2 hn)) with hn = rmsnorm(x, mlp_norm)."""
    H, Hq, Hkv, D, F = 256, 4, 2, 64, 384
    dims = {"H": H, "Hq": Hq, "Hkv": Hkv, "D": D, "F": F, "S_max": 9}
    w = {"attn_norm": gen.normal_f16(3, 0, (H,), 1.0, 0.02), "mlp_norm": gen.normal_f16(3, 1, (H,), 1.0, 0.02),
         "wqkv": gen.workloads.make_layer_weights(_tiny_layer()[0])["wqkv"], "wo": _zero_w4(H, Hq * D),
         "wgate": _diag_w4(F, H, 1.0), "wup": _diag_w4(F, H, 2.0), "wdown": _diag_w4(H, F, 1.0)}
    T, P = 4, 5
    x = gen.normal_f16(4, 0, (T, H))
    kc = np.zeros((Hkv, P + T, D), np.uint16)
    vc = np.zeros((Hkv, P + T, D), np.uint16)
    kc[:, :P] = gen.normal_f16(4, 1, (Hkv, P, D))
    vc[:, :P] = gen.normal_f16(4, 2, (Hkv, P, D))
    out = oracle.verify_layer(dims, w, kc, vc, x, P, np.array([-1, 0, 1, 1], np.int32))
    hn = f64(oracle.rmsnorm(x, w["mlp_norm"]))
    m = f64(f16bits(hn / (1 + np.exp(-hn)) * (2 * hn)))
    assert np.array_equal(out, f16bits(f64(x) + m))


@pytest.mark.parametrize("name", ["c1"])
def test_layer_equals_composition_of_its_stages(name):
    """The one-call reference layer and the stage-by-stage reference chain
    (used for the GPU stage parity) are the same computation, bit for bit."""
    from layer_stages import oracle_stages
    from gen.workloads import CONFIGS, make_activations, make_kv_prefix, make_layer_weights, make_tree
    cfg = CONFIGS[name]
    s = cfg.shape
    w = make_layer_weights(cfg)
    kc, vc = make_kv_prefix(cfg)
    x = make_activations(cfg)
    parent, _ = make_tree(cfg)
    dims = {"H": s.H, "Hq": s.Hq, "Hkv": s.Hkv, "D": s.D, "F": s.F, "S_max": cfg.S_max}
    k1, v1 = kc.copy(), vc.copy()
    out = oracle.verify_layer(dims, w, k1, v1, x, cfg.P, parent)
    k2, v2 = kc.copy(), vc.copy()
    r = oracle_stages(cfg, w, k2, v2, x, parent)
    assert np.array_equal(out, r["out"])
    assert np.array_equal(k1, k2) and np.array_equal(v1, v2)
