"""Pins of the oracle's draft-model attention with a non-square mask
(Sec. 3.1, Fig. 4).  CPU only.

The central pin ties it to the target-model attention, a separately written
function pinned by its own closed forms: expanding the last w nodes of a
tree (all leaves) over a cache that holds the other nodes' rotated rows must
give exactly the target attention's outputs and cache rows for those nodes."""
import numpy as np
import pytest

import gen
import oracle


def _tree_with_leaf_tail(rng, T, w):
    """Increasing tree whose last w nodes are leaves (children of the first T - w)."""
    head = T - w
    parent = [-1] + [int(rng.integers(0, i)) for i in range(1, head)]
    parent += [int(rng.integers(0, head)) for _ in range(w)]
    return np.array(parent, np.int32)


@pytest.mark.parametrize("T,w,D,seed", [(6, 4, 64, 0), (9, 1, 64, 1), (12, 5, 32, 2), (3, 2, 16, 3)])
def test_equals_target_attention_on_leaves(T, w, D, seed):
    rng = np.random.default_rng(seed)
    Hq, Hkv, P = 4, 2, 7
    S_max = P + T + 2
    parent = _tree_with_leaf_tail(rng, T, w)
    q = gen.normal_f16(seed, 1, (T, Hq * D))
    k = gen.normal_f16(seed, 2, (T, Hkv * D))
    v = gen.normal_f16(seed, 3, (T, Hkv * D))
    kc = np.zeros((Hkv, S_max, D), np.uint16)
    kc[:, :P] = gen.normal_f16(seed, 4, (Hkv, P, D))
    vc = kc.copy()
    vc[:, :P] = gen.normal_f16(seed, 5, (Hkv, P, D))
    tk, tv = kc.copy(), vc.copy()
    ref = oracle.tree_attention(q, k, v, tk, tv, P, parent, Hq, Hkv, D)
    # the draft cache: prefix + the target's rotated rows of the first T - w nodes
    N = T - w
    dk, dv = kc.copy(), vc.copy()
    dk[:, P:P + N], dv[:, P:P + N] = tk[:, P:P + N], tv[:, P:P + N]
    out = oracle.draft_tree_attention(q[N:], k[N:], v[N:], dk, dv, P, parent[:N], parent[N:], Hq, Hkv, D)
    assert np.array_equal(out, ref[N:])
    assert np.array_equal(dk, tk) and np.array_equal(dv, tv)


def test_empty_tree_cache_is_single_token_decode():
    D, Hq, Hkv, P, w = 32, 4, 2, 9, 3
    q = gen.normal_f16(7, 1, (w, Hq * D))
    k = gen.normal_f16(7, 2, (w, Hkv * D))
    v = gen.normal_f16(7, 3, (w, Hkv * D))
    kc = np.zeros((Hkv, P + w, D), np.uint16)
    kc[:, :P] = gen.normal_f16(7, 4, (Hkv, P, D))
    vc = kc.copy()
    out = oracle.draft_tree_attention(q, k, v, kc, vc, P, [], [-1] * w, Hq, Hkv, D)
    for i in range(w):
        k1 = np.zeros((Hkv, P + 1, D), np.uint16)
        k1[:, :P] = kc[:, :P]
        v1 = k1.copy()
        v1[:, :P] = vc[:, :P]
        r = oracle.tree_attention(q[i:i + 1], k[i:i + 1], v[i:i + 1], k1, v1, P, [-1], Hq, Hkv, D)
        assert np.array_equal(out[i], r[0])
        assert np.array_equal(kc[:, P + i], k1[:, P])


def test_rows_off_the_root_path_do_not_matter():
    D, Hq, Hkv, P, N, w = 32, 2, 1, 5, 7, 3
    cp = np.array([-1, 0, 0, -1, 3, 1, 2], np.int32)
    lp = np.array([5, 4, -1], np.int32)               # paths: {5,1,0}, {4,3}, {}
    q = gen.normal_f16(8, 1, (w, Hq * D))
    k = gen.normal_f16(8, 2, (w, Hkv * D))
    v = gen.normal_f16(8, 3, (w, Hkv * D))
    kc = gen.normal_f16(8, 4, (Hkv, P + N + w, D))
    vc = gen.normal_f16(8, 5, (Hkv, P + N + w, D))
    base = oracle.draft_tree_attention(q, k, v, kc.copy(), vc.copy(), P, cp, lp, Hq, Hkv, D)
    for row in range(N):
        k2, v2 = kc.copy(), vc.copy()
        k2[:, P + row] = gen.normal_f16(9, row, (Hkv, D))
        v2[:, P + row] = gen.normal_f16(10, row, (Hkv, D))
        out = oracle.draft_tree_attention(q, k, v, k2, v2, P, cp, lp, Hq, Hkv, D)
        for i, path in enumerate(({5, 1, 0}, {4, 3}, set())):
            same = np.array_equal(out[i], base[i])
            assert same == (row not in path), (row, i)


def test_invalid_arguments_rejected():
    q = np.zeros((1, 64), np.uint16)
    kv = np.zeros((1, 32), np.uint16)
    kc = np.zeros((1, 20, 32), np.uint16)
    with pytest.raises(ValueError):
        oracle.draft_tree_attention(q, kv, kv, kc, kc.copy(), 5, [-1, 2], [0], 2, 1, 32)   # bad forest
    with pytest.raises(ValueError):
        oracle.draft_tree_attention(q, kv, kv, kc, kc.copy(), 5, [-1], [1], 2, 1, 32)      # leaf parent
    with pytest.raises(ValueError):
        oracle.draft_tree_attention(q, kv, kv, kc, kc.copy(), 19, [-1], [0], 2, 1, 32)     # no room
