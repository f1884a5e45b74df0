"""Pins of the oracle's draft-tree bookkeeping (Sec. 3.1: Alg. 1 and the
maximum-likelihood tree expansion; Sec. 3.2 / Fig. 5 for re-rooting) and of
its top-k log-softmax (the children of an expanded leaf).  CPU only."""
import itertools
import math
import os

import numpy as np
import pytest

import oracle
from oracle.draft_tree import DraftTree

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _from_nodes(nodes):
    """A DraftTree built from (token, parent index, value) in index order;
    nodes with children are expanded and own tree-cache rows in index
    order (the root excepted)."""
    t = DraftTree(nodes[0][0])
    for tok, par, val in nodes[1:]:
        t.token.append(tok)
        t.parent.append(par)
        t.value.append(val)
        t.weight.append(t.weight[par] + val)
        t.expanded.append(False)
        t.selected.append(False)
        t.row.append(-1)
    for i in range(t.size()):
        if t.children(i):
            t.expanded[i] = True
            if i:
                t.row[i] = t.n_rows
                t.n_rows += 1
    return t


def _random_tree(rng, n_rounds, w, k, vocab=50):
    t = DraftTree(int(rng.integers(vocab)))
    for _ in range(n_rounds):
        leaves, _ = t.select_leaves(w)
        if not leaves:
            break
        toks, lps = [], []
        for _ in leaves:
            p = rng.dirichlet(np.full(vocab, 0.3))
            top = np.argsort(-p, kind="stable")[:k]
            toks.append([int(x) for x in top])
            lps.append([math.log(p[x]) for x in top])
        t.expand(leaves, toks, lps)
    return t


def _path_prob(t, v):
    """Product of the node probabilities from the root to v (independent of
    the summed weights)."""
    pr = 1.0
    while v > 0:
        pr *= math.exp(t.value[v])
        v = t.parent[v]
    return pr


# ------------------------------------------------------------- golden
def _read_fig3():
    nodes, steps = [], []
    for line in open(os.path.join(GOLD, "fig3_tree_generation.txt")):
        f = line.split("#")[0].split()
        if not f:
            continue
        if f[0] == "node":
            nodes.append((int(f[1]), None if f[2] == "-" else int(f[2]), float(f[3])))
        elif f[0] != "tree":
            steps.append((f[0], [int(x) for x in f[1:]]))
    return nodes, steps


def test_fig3_tree_generation_walkthrough():
    nodes, steps = _read_fig3()
    idx = {tok: i for i, (tok, _, _) in enumerate(nodes)}
    full = [(tok, -1 if par is None else idx[par], val) for tok, par, val in nodes]
    initial = [n for n in full if n[0] <= 6]
    t = _from_nodes(full)
    for kind, args in steps:
        if kind == "subgraph_initial":
            _, _, toks = _from_nodes(initial).select_subgraph(args[0])
            assert toks == args[1:]
        elif kind == "subgraph":
            _, par, toks = t.select_subgraph(args[0])
            assert toks == args[1:] and par[0] == -1
        elif kind == "verified":
            r = t.reroot(args)
        elif kind == "expect_root":
            assert t.token[0] == args[0]
        elif kind == "expect_tree":
            assert t.token == args
    # the second output ends outside the tree: t16 is a fresh, pending root,
    # behind t9 whose keys and values the draft already holds
    assert r["keep"] == 0 and r["pending"] == [16]


def test_fig5_reroot_matches_kv_update():
    """Sec. 3.2 / Fig. 5: the tree cache below t10; verified (t12, t15) keep
    t15's subtree t17, t18, and the rows the tree manager reports agree with
    the KV reorganisation of the same example."""
    rows = []
    for line in open(os.path.join(GOLD, "fig5_kv_update.txt")):
        f = line.split("#")[0].split()
        if f and f[0] == "node":
            rows.append((int(f[1]), int(f[2])))
        if f and f[0] == "expect_tree":
            expect_tree = [int(x) for x in f[1:]]
        if f and f[0] == "expect_parent":
            expect_parent = [int(x) for x in f[1:]]
    # root t10 (the last prefix token), tree-cache row r = node r + 1
    nodes = [(10, -1, 0.0)] + [(tok, 0 if pr < 0 else pr + 1, -0.1) for tok, pr in rows]
    t = _from_nodes(nodes)
    # every fixture row is a tree-cache row, in fixture order
    for r in range(len(rows)):
        t.expanded[r + 1] = True
        t.row[r + 1] = r
    t.n_rows = len(rows)
    forest = t.forest()
    assert forest == [p for _, p in rows]
    res = t.reroot([10, 12, 15])
    assert res == {"last": 4, "path_rows": 2, "keep": 1, "pending": []}
    assert t.token == [15] + expect_tree
    assert t.forest() == expect_parent
    # the same rows through the oracle's KV reorganisation
    P, N, D = 4, len(rows), 8
    kc = np.zeros((1, 16, D), np.uint16)
    kc[0, P:P + N, 0] = [tok for tok, _ in rows]
    vc = kc.copy()
    L, new_parent = oracle.kv_reorganize(kc, vc, P, np.array(forest, np.int32), res["last"], keep=True)
    n_kept = len(new_parent)
    assert L == res["path_rows"] and n_kept == t.n_rows and list(new_parent) == t.forest()
    assert list(kc[0, P + L:P + L + n_kept, 0]) == t.token[1:]


# ------------------------------------------------------- brute force
@pytest.mark.parametrize("seed", range(6))
def test_subgraph_is_most_probable_connected_set(seed):
    """The selected bs nodes maximise the summed path probability over every
    connected node set of size bs that contains the root (the expected
    number of tokens the draft distribution would accept)."""
    rng = np.random.default_rng(seed)
    t = _random_tree(rng, n_rounds=3, w=2, k=2, vocab=12)
    n = t.size()
    prob = [_path_prob(t, v) for v in range(n)]
    for bs in (1, 2, 3, 4, 5):
        if bs > n:
            break
        best, best_set = -1.0, None
        for rest in itertools.combinations(range(1, n), bs - 1):
            s = {0, *rest}
            if all(t.parent[v] in s for v in rest):
                tot = sum(prob[v] for v in s)
                if tot > best + 1e-15:
                    best, best_set = tot, sorted(s)
        nodes, parent, toks = t.select_subgraph(bs)
        assert nodes == best_set
        assert parent[0] == -1 and all(0 <= parent[j] < j for j in range(1, bs))


@pytest.mark.parametrize("seed", range(6))
def test_expansion_takes_most_probable_leaves(seed):
    rng = np.random.default_rng(100 + seed)
    t = _random_tree(rng, n_rounds=4, w=3, k=3, vocab=20)
    open_ = [v for v in range(t.size()) if not t.expanded[v]]
    expect = sorted(open_, key=lambda v: -_path_prob(t, v))[:3]
    got, prow = t.select_leaves(3)
    assert sorted(got) == sorted(expect)
    assert [_path_prob(t, v) for v in got] == sorted((_path_prob(t, v) for v in got), reverse=True)
    for v, pr in zip(got, prow):
        assert pr == (-1 if t.parent[v] == 0 else t.row[t.parent[v]])


@pytest.mark.parametrize("seed", range(8))
def test_reroot_keeps_exactly_the_subtree(seed):
    """Re-rooting on a path ending at an expanded node keeps that node's
    subtree: the same token paths below it, the same path probabilities
    relative to it, tree-cache rows in their old order, and a forest equal
    to the one the KV reorganisation produces."""
    rng = np.random.default_rng(200 + seed)
    t = _random_tree(rng, n_rounds=5, w=2, k=2, vocab=10)
    exp_nodes = [v for v in range(1, t.size()) if t.expanded[v]]
    end = exp_nodes[int(rng.integers(len(exp_nodes)))]
    path = []
    v = end
    while v >= 0:
        path.append(v)
        v = t.parent[v]
    path = path[::-1]
    verified = [t.token[v] for v in path]

    def seqs(tree, root):
        out = {}
        for v in range(tree.size()):
            s, u = [], v
            while u != root and u >= 0:
                s.append(tree.token[u])
                u = tree.parent[u]
            if u == root:
                out[tuple(s[::-1])] = _path_prob(tree, v) / _path_prob(tree, root)
        return out

    before = seqs(t, end)
    old_rows = {v: t.row[v] for v in range(t.size())}
    sub = [v for v in range(t.size()) if t._below_or_at(v, end)]
    forest = t.forest()
    res = t.reroot(verified)
    assert res["keep"] == 1 and res["pending"] == []
    assert res["last"] == old_rows[end] and res["path_rows"] == len(path) - 1
    after = seqs(t, 0)
    for v in range(t.size()):  # weights are relative to the new root
        assert math.isclose(math.exp(t.weight[v]), _path_prob(t, v), rel_tol=1e-12)
    assert before.keys() == after.keys()
    for key in before:
        assert math.isclose(before[key], after[key], rel_tol=1e-12)
    kept_old_rows = sorted(old_rows[v] for v in sub if v != end and old_rows[v] >= 0)
    assert t.n_rows == len(kept_old_rows)
    P, D = 3, 8
    kc = np.zeros((1, P + len(forest) + 2, D), np.uint16)
    kc[0, P:P + len(forest), 0] = np.arange(1, len(forest) + 1)
    vc = kc.copy()
    L, new_parent = oracle.kv_reorganize(kc, vc, P, np.array(forest, np.int32), res["last"], keep=True)
    n_kept = len(new_parent)
    assert L == res["path_rows"] and n_kept == t.n_rows and list(new_parent) == t.forest()
    assert list(kc[0, P + L:P + L + n_kept, 0]) == [r + 1 for r in kept_old_rows]


def test_reroot_off_tree_and_unexpanded_end():
    t = DraftTree(5)
    leaves, _ = t.select_leaves(1)
    t.expand(leaves, [[7, 8]], [[-0.1, -1.0]])
    leaves, _ = t.select_leaves(1)
    t.expand(leaves, [[2]], [[-0.1]])
    # 7 (expanded) then 2 (a leaf without keys/values) then 9 (not in the tree)
    res = t.reroot([5, 7, 2, 9])
    assert res == {"last": 0, "path_rows": 1, "keep": 0, "pending": [2, 9]}
    assert t.token == [9] and not t.expanded[0]
    # a pending root: the next re-root also reports the root itself
    res = t.reroot([9, 4])
    assert res == {"last": -1, "path_rows": 0, "keep": 0, "pending": [9, 4]}
    with pytest.raises(AssertionError):
        t.reroot([3, 1])
    with pytest.raises(AssertionError):  # an output holds at least the root and one token
        t.reroot([4])


# ------------------------------------------------------------ top-k
def _f16(x):
    return np.asarray(x, np.float16).view(np.uint16)


def test_topk_closed_forms():
    V = 1000
    # equal logits: -log V each, the lowest indices
    tok, lp = oracle.topk_logprobs(_f16(np.full((1, V), 0.75)), 4)
    assert list(tok[0]) == [0, 1, 2, 3]
    assert np.allclose(lp, -math.log(V), atol=1e-12)
    # one logit a above V - 1 logits b: log p = -log(1 + (V-1) e^(b-a))
    x = np.full((1, V), -1.0)
    x[0, 417] = 2.5
    tok, lp = oracle.topk_logprobs(_f16(x), 2)
    assert list(tok[0]) == [417, 0]
    assert math.isclose(lp[0, 0], -math.log1p((V - 1) * math.exp(-3.5)), rel_tol=1e-12)
    assert math.isclose(lp[0, 1], -3.5 - math.log1p((V - 1) * math.exp(-3.5)), rel_tol=1e-12)


def test_topk_against_full_softmax_and_sort():
    rng = np.random.default_rng(7)
    # multiples of 1/64 below 12 in magnitude: shifting by 4 stays exact in fp16
    x = _f16(np.clip(np.round(rng.standard_normal((5, 300)) * 3 * 64) / 64, -11.5, 11.5))
    x[2, 10:20] = x[2, 5]  # planted ties
    tok, lp = oracle.topk_logprobs(x, 8)
    xf = x.view(np.float16).astype(np.float64)
    for i in range(5):
        order = sorted(range(300), key=lambda v: (-xf[i, v], v))[:8]
        assert list(tok[i]) == order
        p = np.exp(xf[i] - xf[i].max())
        p /= p.sum()
        assert np.allclose(np.exp(lp[i]), p[order], rtol=1e-12)
    # shift invariance
    tok2, lp2 = oracle.topk_logprobs(_f16(xf + 4.0), 8)
    assert np.array_equal(tok, tok2) and np.allclose(lp, lp2, atol=1e-12)
