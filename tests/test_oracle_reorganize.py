"""Pins of the oracle's draft-side KV reorganisation (Sec. 3.2, consistency
management of the draft model's cache; Fig. 5).  CPU only."""
import itertools
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "fig5_kv_update.txt")


def _caches(P, N, extra, Hkv=2, D=8, n_layers=1, seed=0):
    """Caches whose row r of head g, layer l holds a recognisable pattern."""
    S_max = P + N + extra
    rng = np.random.default_rng(seed)
    k = rng.integers(0, 65535, (n_layers, Hkv, S_max, D)).astype(np.uint16)
    v = rng.integers(0, 65535, (n_layers, Hkv, S_max, D)).astype(np.uint16)
    return k, v


def test_fig5_example():
    prefix, nodes, verified, exp = [], [], [], {}
    for line in open(GOLDEN):
        f = line.split("#")[0].split()
        if not f:
            continue
        if f[0] == "prefix":
            prefix = [int(t) for t in f[1:]]
        elif f[0] == "node":
            nodes.append((int(f[1]), int(f[2])))
        elif f[0] == "verified":
            verified = [int(t) for t in f[1:]]
        else:
            exp[f[0]] = [int(t) for t in f[1:]]
    tok = [t for t, _ in nodes]
    parent = np.array([p for _, p in nodes], np.int32)
    P, N = len(prefix), len(nodes)
    # walk the forest with the verified tokens: the deepest node reached
    last, here = -1, -1
    for t in verified:
        nxt = [c for c in range(N) if parent[c] == here and tok[c] == t]
        if not nxt:
            break
        here = last = nxt[0]
    # one head, one column: a cache row holds its token id
    k = np.zeros((1, 1, P + N + 2, 8), np.uint16)
    k[0, 0, :P, 0] = prefix
    k[0, 0, P:P + N, 0] = tok
    v = k.copy()
    L, newp = oracle.kv_reorganize(k, v, P, parent, last, keep=True)
    assert list(k[0, 0, :P + L, 0]) == exp["expect_prefix"]
    assert list(k[0, 0, P + L:P + L + len(newp), 0]) == exp["expect_tree"]
    assert list(newp) == exp["expect_parent"]
    assert np.array_equal(k, v)


def _brute(P, parent, last, keep, k):
    """Rows after the update, by definition: the path (forest root .. last)
    then, if kept, every node having last as a proper ancestor, in index
    order."""
    N = len(parent)
    anc = [set() for _ in range(N)]
    for c in range(N):
        j = parent[c]
        while j != -1:
            anc[c].add(j)
            j = parent[j]
    path = sorted((anc[last] | {last}) if last >= 0 else set())
    kept = [c for c in range(N) if keep and last >= 0 and last in anc[c]]
    out = k.copy()
    for i, src in enumerate(path + kept):
        out[..., P + i, :] = k[..., P + src, :]
    newp = [kept.index(parent[c]) if parent[c] != last else -1 for c in kept]
    return out, len(path), newp


def _forests(N):
    for par in itertools.product(*[range(-1, i) for i in range(N)]):
        yield np.array(par, np.int32)


@pytest.mark.parametrize("N", [1, 2, 3, 4, 5])
def test_all_small_forests(N):
    P = 3
    for parent in _forests(N):
        for last in range(-1, N):
            for keep in (False, True):
                k, v = _caches(P, N, 2, seed=N)
                ref, L0, newp0 = _brute(P, list(parent), last, keep, k)
                L, newp = oracle.kv_reorganize(k, v, P, parent, last, keep)
                assert L == L0 and list(newp) == newp0
                assert np.array_equal(k, ref)
                assert all(p < j for j, p in enumerate(newp))   # still a forest in index order


def test_without_subtree_equals_target_commit():
    """keep = False on a single-root tree is the target model's commit."""
    rng = np.random.default_rng(3)
    for trial in range(30):
        T = int(rng.integers(1, 12))
        parent = np.array([-1] + [int(rng.integers(0, i)) for i in range(1, T)], np.int32)
        acc = int(rng.integers(0, T))
        k, v = _caches(5, T, 3, n_layers=2, seed=trial)
        k2, v2 = k.copy(), v.copy()
        L, newp = oracle.kv_reorganize(k, v, 5, parent, acc, keep=False, n_layers=2)
        L2 = oracle.kv_commit(k2, v2, 5, parent, acc, n_layers=2)
        assert L == L2 and len(newp) == 0
        assert np.array_equal(k, k2) and np.array_equal(v, v2)


def test_special_cases():
    k, v = _caches(4, 6, 1)
    k0 = k.copy()
    # nothing verified inside the forest: nothing moves
    L, newp = oracle.kv_reorganize(k, v, 4, [-1, 0, 0, -1, 3, 4], -1, True)
    assert L == 0 and len(newp) == 0 and np.array_equal(k, k0)
    # a root with everything below it: the whole forest under it shifts by one
    k, v = _caches(4, 6, 1)
    k0 = k.copy()
    L, newp = oracle.kv_reorganize(k, v, 4, [-1, 0, 0, 1, 3, 2], 0, True)
    assert L == 1 and list(newp) == [-1, -1, 0, 2, 1]
    assert np.array_equal(k[..., 4:10, :], k0[..., 4:10, :])
    # invalid forest rejected
    with pytest.raises(ValueError):
        oracle.kv_reorganize(k, v, 4, [-1, 2, 0], 0, True)
