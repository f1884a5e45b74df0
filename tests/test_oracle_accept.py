"""Pins of the oracle's greedy acceptance (target-side verification with the
target's greedy choice; Sec. 3.1, Fig. 3 walk-through).  CPU only."""
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "fig3_walkthrough.txt")


def _logits_choosing(choices, V, seed):
    """fp16 logits [T][V] whose row maxima sit exactly at `choices`: N(0, 1)
    draws clipped below 4, then 8.0 at the chosen index."""
    rng = np.random.default_rng(seed)
    x = np.minimum(rng.standard_normal((len(choices), V)), 4.0)
    x[np.arange(len(choices)), choices] = 8.0
    return x.astype(np.float16).view(np.uint16)


def _read_golden():
    iters, outputs = {}, {}
    for line in open(GOLDEN):
        line = line.split("#")[0].split()
        if not line:
            continue
        if line[0] == "output":
            outputs[int(line[1])] = [int(t) for t in line[2:]]
        else:
            it, node, tok, par, nxt = map(int, line)
            iters.setdefault(it, []).append((node, tok, par, nxt))
    return iters, outputs


def test_fig3_walkthrough():
    iters, outputs = _read_golden()
    assert sorted(iters) == sorted(outputs) == [1, 2]
    for it, rows in iters.items():
        rows.sort()
        tokens = np.array([r[1] for r in rows], np.int32)
        parent = np.array([r[2] for r in rows], np.int32)
        choices = np.array([r[3] for r in rows])
        logits = _logits_choosing(choices, 32, it)
        am, acc, bonus, L = oracle.greedy_accept(logits, tokens, parent)
        assert np.array_equal(am, choices)
        path = []
        j = acc
        while j != -1:
            path.append(int(tokens[j]))
            j = int(parent[j])
        assert path[::-1] + [bonus] == outputs[it]
        assert L == len(path)


def test_argmax_is_first_maximum():
    """Row choice against numpy's argmax (first occurrence) on fp16 logits
    with planted ties, including all-equal rows and negative rows."""
    rng = np.random.default_rng(5)
    T, V = 12, 1000
    x = rng.standard_normal((T, V)).astype(np.float16)
    x[1, [17, 400, 999]] = np.float16(9.0)       # three-way tie
    x[2, :] = np.float16(0.25)                   # all equal: index 0
    x[3] = -np.abs(x[3]) - np.float16(1.0)       # all negative
    x[4, [0, 999]] = np.float16(7.5)             # tie at both ends
    x[5, 600] = np.float16(65504.0)              # largest finite
    parent = np.concatenate([[-1], np.arange(T - 1)]).astype(np.int32)
    tokens = np.full(T, -5, np.int32)
    am, acc, bonus, L = oracle.greedy_accept(x.view(np.uint16), tokens, parent)
    assert np.array_equal(am, np.argmax(x.astype(np.float64), axis=1))
    assert am[1] == 17 and am[2] == 0 and am[4] == 0 and am[5] == 600
    assert (acc, bonus, L) == (0, am[0], 1)


def _accepted_by_characterisation(parent, tokens, am):
    """The accepted node as the unique node whose root path is consistent
    (every step goes to the smallest-index child carrying the parent's
    choice) and none of whose children is consistent."""
    T = len(parent)

    def step_ok(c):
        p = parent[c]
        if tokens[c] != am[p]:
            return False
        return all(not (parent[d] == p and tokens[d] == am[p]) for d in range(1, c))

    consistent = []
    for i in range(T):
        j, ok = i, True
        while parent[j] != -1:
            ok = ok and step_ok(j)
            j = parent[j]
        if ok:
            consistent.append(i)
    leaves = [i for i in consistent if not any(parent[c] == i for c in consistent)]
    assert len(leaves) == 1
    return leaves[0]


@pytest.mark.parametrize("seed", range(40))
def test_walk_matches_characterisation(seed):
    rng = np.random.default_rng(100 + seed)
    T = int(rng.integers(1, 11))
    parent = np.array([-1] + [int(rng.integers(0, i)) for i in range(1, T)], np.int32)
    vocab = int(rng.integers(1, 4))                # few tokens: many matches and sibling ties
    tokens = rng.integers(0, vocab, T).astype(np.int32)
    choices = rng.integers(0, vocab, T)
    logits = _logits_choosing(choices, 8, seed)
    am, acc, bonus, L = oracle.greedy_accept(logits, tokens, parent)
    assert np.array_equal(am, choices)
    assert acc == _accepted_by_characterisation(list(parent), list(tokens), list(am))
    assert bonus == am[acc]
    depth, _ = oracle.tree(parent)
    assert L == depth[acc] + 1


def test_special_cases():
    V = 16
    # single node: the root is accepted and the bonus is its choice
    am, acc, bonus, L = oracle.greedy_accept(_logits_choosing([5], V, 1), np.array([3], np.int32),
                                             np.array([-1], np.int32))
    assert (acc, bonus, L) == (0, 5, 1)
    # chain whose tokens all match: every node accepted
    T = 7
    parent = np.arange(-1, T - 1, dtype=np.int32)
    choices = np.arange(1, T + 1)
    tokens = np.arange(0, T, dtype=np.int32)
    am, acc, bonus, L = oracle.greedy_accept(_logits_choosing(choices, V, 2), tokens, parent)
    assert (acc, bonus, L) == (T - 1, T, T)
    # nothing matches: the root alone
    am, acc, bonus, L = oracle.greedy_accept(_logits_choosing(np.full(T, 15), V, 3), tokens, parent)
    assert (acc, bonus, L) == (0, 15, 1)
    # two siblings carry the chosen token: the lower index wins
    parent = np.array([-1, 0, 0, 0, 2, 1], np.int32)
    tokens = np.array([0, 4, 9, 9, 1, 1], np.int32)
    choices = np.array([9, 0, 1, 0, 0, 0])
    am, acc, bonus, L = oracle.greedy_accept(_logits_choosing(choices, V, 4), tokens, parent)
    assert (acc, bonus, L) == (4, 0, 3)


def test_invalid_tree_rejected():
    with pytest.raises(ValueError):
        oracle.greedy_accept(_logits_choosing([1, 2], 4, 0), np.array([0, 0], np.int32),
                             np.array([-1, 1], np.int32))
