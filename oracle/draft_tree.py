"""Draft-tree bookkeeping of parallel tree generation -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use this module; the product path never imports it.

Plain Python, slow and direct: lists indexed by node, full sorts where the
product keeps a priority queue.  It follows Sec. 3.1 (Alg. 1, parallel tree
generation, and the maximum-likelihood tree expansion paragraph) for the tree
and Sec. 3.2 (KV-cache consistency management, Fig. 5) for the draft cache
rows:

* A node's value is the log-softmax probability of its token under the draft
  distribution of its parent; its weight is the sum of values from the root
  to the node (the root's weight is 0), accumulated in double precision as
  ``weight[parent] + value``.
* Ordering: a larger weight first, then the lower node index.  Values are
  log-probabilities (<= 0), so a child never precedes its parent.
* Expansion runs the draft model on the w unexpanded nodes that come first
  in that order; each gets the k most probable children (appended in leaf
  order, then child rank) and is marked expanded.
* The draft cache: the root's key/value are the last row of the prefix
  cache; every other expanded node owns one tree-cache row, numbered in the
  order the nodes were selected for expansion.
* The subgraph sent to the target: the bs nodes first in the order, listed by
  node index (parents before children), with parents as positions in that
  list.
* Re-rooting: the verified tokens start with the root's token; the walk goes
  to the child carrying the next verified token while there is one.  The
  forest rows of the walked expanded nodes move to the prefix.  If the walk
  consumed every verified token and ended on an expanded node, that node
  becomes the root and its subtree is kept (renumbered in index order, cache
  rows in row order, weights relative to the new root); otherwise the tree
  restarts from a fresh root carrying the last verified token, and the
  verified tokens whose keys and values the draft has not computed yet are
  returned as pending (they precede the fresh root in the draft's context,
  the root included).
"""
from __future__ import annotations

import math


class DraftTree:
    def __init__(self, root_token: int):
        self.token = [int(root_token)]
        self.parent = [-1]
        self.value = [0.0]
        self.weight = [0.0]
        self.expanded = [False]
        self.selected = [False]
        self.row = [-1]
        self.n_rows = 0

    # ---------------------------------------------------------------- queries
    def size(self) -> int:
        return len(self.token)

    def children(self, i: int):
        return [j for j in range(self.size()) if self.parent[j] == i]

    def key(self, i: int):
        return (-self.weight[i], i)

    def forest(self):
        """Parent row of every tree-cache row (-1: below the root, the last
        prefix row)."""
        out = [0] * self.n_rows
        for i in range(1, self.size()):
            if self.row[i] >= 0:
                p = self.parent[i]
                out[self.row[i]] = self.row[p] if p != 0 else -1
        return out

    # -------------------------------------------------------------- expansion
    def select_leaves(self, w: int):
        """The up to w unexpanded, unselected nodes first in the order; each
        non-root one gets the next tree-cache row.  Returns (nodes, parent
        row of each: -1 below the root)."""
        cand = [i for i in range(self.size()) if not self.expanded[i] and not self.selected[i]]
        cand.sort(key=self.key)
        out = cand[:w]
        prow = []
        for i in out:
            self.selected[i] = True
            if i != 0:
                self.row[i] = self.n_rows
                self.n_rows += 1
            p = self.parent[i]
            prow.append(-1 if p <= 0 else self.row[p])
        return out, prow

    def expand(self, leaves, tokens, logprobs):
        """Children of each selected leaf: tokens[j][c] with value
        logprobs[j][c] (a log-probability: <= 0)."""
        for j, i in enumerate(leaves):
            assert self.selected[i] and not self.expanded[i]
            for c in range(len(tokens[j])):
                lp = float(logprobs[j][c])
                assert lp <= 0.0 and not math.isnan(lp)
                self.token.append(int(tokens[j][c]))
                self.parent.append(i)
                self.value.append(lp)
                self.weight.append(self.weight[i] + lp)
                self.expanded.append(False)
                self.selected.append(False)
                self.row.append(-1)
            self.expanded[i] = True
            self.selected[i] = False

    # ---------------------------------------------------------------- subgraph
    def select_subgraph(self, bs: int):
        """(nodes, parent positions, tokens) of the bs nodes first in the
        order, listed by node index."""
        top = sorted(range(self.size()), key=self.key)[:bs]
        nodes = sorted(top)
        pos = {v: j for j, v in enumerate(nodes)}
        parent = [-1 if v == 0 else pos[self.parent[v]] for v in nodes]
        return nodes, parent, [self.token[v] for v in nodes]

    # ---------------------------------------------------------------- re-root
    def reroot(self, verified):
        """Walk the verified tokens from the root and re-root.  Returns a dict:
        last (tree-cache row of the deepest walked expanded node, -1 if
        none), path_rows (rows that move to the prefix), keep (1 if the
        subtree below `last` is kept), pending (tokens whose draft keys and
        values are still to be computed, in context order)."""
        verified = [int(t) for t in verified]
        # an output holds the root and at least the token after it
        assert len(verified) >= 2 and verified[0] == self.token[0]
        assert not any(self.selected)
        walked = [0]
        for t in verified[1:]:
            nxt = [c for c in self.children(walked[-1]) if self.token[c] == t]
            if not nxt:
                break
            walked.append(nxt[0])
        assert len(walked) >= len(verified) - 1, "a verified token before the last is not in the tree"
        rows = [self.row[v] for v in walked[1:] if self.row[v] >= 0]
        last = rows[-1] if rows else -1
        end = walked[-1]
        keep = len(walked) == len(verified) and end != 0 and self.expanded[end]
        if keep:
            sub = [v for v in range(self.size()) if self._below_or_at(v, end)]
            kept_rows = sorted(self.row[v] for v in sub if v != end and self.row[v] >= 0)
            rowmap = {r: j for j, r in enumerate(kept_rows)}
            idx = {v: j for j, v in enumerate(sub)}
            base = self.weight[end]
            self.token = [self.token[v] for v in sub]
            self.parent = [-1 if v == end else idx[self.parent[v]] for v in sub]
            self.value = [0.0 if v == end else self.value[v] for v in sub]
            self.weight = [self.weight[v] - base for v in sub]
            self.expanded = [self.expanded[v] for v in sub]
            self.selected = [False] * len(sub)
            self.row = [-1 if v == end or self.row[v] < 0 else rowmap[self.row[v]] for v in sub]
            self.n_rows = len(kept_rows)
            return {"last": last, "path_rows": len(rows), "keep": 1, "pending": []}
        # the draft has keys and values for the root (if expanded) and the
        # walked expanded nodes; the remaining verified tokens are pending
        first = 1 + len(rows)
        pending = ([] if self.expanded[0] else [self.token[0]]) + verified[first:]
        self.__init__(verified[-1])
        return {"last": last, "path_rows": len(rows), "keep": 0, "pending": pending}

    def _below_or_at(self, v: int, a: int) -> bool:
        while v >= 0:
            if v == a:
                return True
            v = self.parent[v]
        return False
