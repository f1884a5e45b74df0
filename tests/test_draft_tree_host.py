"""The library's host-side draft tree (swiftspec_draft_tree_*) against the
oracle's, operation by operation (Sec. 3.1, Alg. 1 and the maximum-
likelihood expansion; re-rooting per Sec. 3.2).  Host code only: runs on
the CPU."""
import math

import numpy as np
import pytest

import paper_2506_11309_amd as ss
from oracle.draft_tree import DraftTree as OracleTree


def _children_dist(rng, k, vocab):
    """k distinct tokens with float32 log-probabilities (non-increasing)."""
    p = rng.dirichlet(np.full(vocab, 0.2))
    top = np.argsort(-p, kind="stable")[:k]
    lp = np.log(np.maximum(p[top], 1e-30)).astype(np.float32)
    return top.astype(np.int32), np.minimum(lp, 0).astype(np.float32)


def _same(lib, orc):
    tok, par, w, row, exp = lib.nodes()
    assert list(tok) == orc.token
    assert list(par) == orc.parent
    assert list(w) == orc.weight  # bit-identical doubles: same sums in the same order
    assert list(row) == orc.row
    assert [bool(x) for x in exp] == orc.expanded
    assert lib.rows() == orc.n_rows
    assert list(lib.forest()) == orc.forest()


def _grow(rng, lib, orc, w, k, vocab):
    leaves, prow = lib.select_leaves(w)
    oleaves, oprow = orc.select_leaves(w)
    assert list(leaves) == oleaves and list(prow) == oprow
    if len(leaves) == 0:
        return
    toks, lps = zip(*(_children_dist(rng, k, vocab) for _ in leaves))
    lib.expand(leaves, np.array(toks), np.array(lps))
    orc.expand(oleaves, [list(map(int, t)) for t in toks], [[float(x) for x in l] for l in lps])


def _verified(rng, orc, vocab):
    """A target output: root path to a random node, then a bonus token that
    is a child's token, or absent from the tree."""
    v = int(rng.integers(orc.size()))
    path = []
    while v >= 0:
        path.append(v)
        v = orc.parent[v]
    seq = [orc.token[u] for u in path[::-1]]
    kids = orc.children(path[0])
    r = rng.random()
    if kids and r < 0.6:
        seq.append(orc.token[kids[int(rng.integers(len(kids)))]])
    else:
        seq.append(int(vocab + rng.integers(100)))  # not in the tree
    return seq


@pytest.mark.parametrize("seed", range(12))
def test_loop_matches_oracle(seed):
    """Iterations of the draft worker's loop (Alg. 1): d expansion steps,
    re-rooting on a target output, growing while the tree is smaller than
    bs, the bs-node subgraph -- every output and the whole tree state equal
    the oracle's after every operation."""
    rng = np.random.default_rng(seed)
    vocab, w, k, d, bs = 30, int(rng.integers(1, 5)), int(rng.integers(1, 4)), 3, int(rng.integers(1, 9))
    root = int(rng.integers(vocab))
    lib, orc = ss.DraftTree(4096, root), OracleTree(root)
    _same(lib, orc)
    for it in range(8):
        for _ in range(d):
            _grow(rng, lib, orc, w, k, vocab)
            _same(lib, orc)
        ver = _verified(rng, orc, vocab)
        assert lib.reroot(ver) == orc.reroot(ver)
        _same(lib, orc)
        while orc.size() < bs:
            _grow(rng, lib, orc, w, k, vocab)
            _same(lib, orc)
        nodes, par, tok = lib.select_subgraph(bs)
        onodes, opar, otok = orc.select_subgraph(bs)
        assert list(nodes) == onodes and list(par) == opar and list(tok) == otok


def test_invalid_calls_leave_the_tree_unchanged():
    rng = np.random.default_rng(3)
    lib, orc = ss.DraftTree(16, 7), OracleTree(7)
    _grow(rng, lib, orc, 1, 3, 20)
    before = lib.nodes()
    leaves, _ = lib.select_leaves(2)
    orc.select_leaves(2)
    with pytest.raises(ss.SwiftSpecError) as e:  # a log-probability above 0
        lib.expand(leaves, np.array([[1], [2]]), np.array([[-0.5], [0.25]], np.float32))
    assert e.value.status == ss.INVALID_ARG
    with pytest.raises(ss.SwiftSpecError) as e:  # NaN
        lib.expand(leaves, np.array([[1], [2]]), np.array([[-0.5], [np.nan]], np.float32))
    with pytest.raises(ss.SwiftSpecError) as e:  # a leaf twice
        lib.expand(np.array([leaves[0], leaves[0]]), np.array([[1], [2]]), np.array([[-0.5], [-1]], np.float32))
    with pytest.raises(ss.SwiftSpecError) as e:  # an unselected node
        lib.expand(np.array([0]), np.array([[1]]), np.array([[-0.5]], np.float32))
    with pytest.raises(ss.SwiftSpecError) as e:  # capacity: 4 nodes + 2 x 7 > 16
        lib.expand(leaves, np.arange(14).reshape(2, 7), np.full((2, 7), -1.0, np.float32))
    assert e.value.status == ss.CAPACITY
    with pytest.raises(ss.SwiftSpecError) as e:  # re-root with selected leaves pending
        lib.reroot([7])
    for a, b in zip(before[:3], lib.nodes()[:3]):
        assert np.array_equal(a, b)
    lib.expand(leaves, np.array([[1], [2]]), np.array([[-0.5], [-1]], np.float32))
    orc.expand(list(leaves), [[1], [2]], [[-0.5], [-1.0]])
    _same(lib, orc)
    with pytest.raises(ss.SwiftSpecError):  # no token after the root
        lib.reroot([7])
    with pytest.raises(ss.SwiftSpecError):  # not the root token
        lib.reroot([8, 1])
    with pytest.raises(ss.SwiftSpecError):  # a middle token off the tree
        lib.reroot([7, 99, 1])
    _same(lib, orc)


def test_large_tree_selection_is_exact():
    """A 3000-node tree (the priority queue and the partial selection at
    scale) equals the oracle's full sorts."""
    rng = np.random.default_rng(11)
    lib, orc = ss.DraftTree(4000, 1), OracleTree(1)
    while orc.size() < 3000:
        _grow(rng, lib, orc, 8, 4, 1000)
    _same(lib, orc)
    for bs in (1, 8, 64, 512):
        nodes, par, _ = lib.select_subgraph(bs)
        onodes, opar, _ = orc.select_subgraph(bs)
        assert list(nodes) == onodes and list(par) == opar
