// Host-side draft tree of parallel tree generation (Sec. 3.1, Alg. 1 and the
// maximum-likelihood tree expansion; re-rooting and draft-cache rows per
// Sec. 3.2 and Fig. 5).
//
// A node's value is the log-probability of its token under its parent's
// draft distribution, its weight the sum of values from the root (double,
// accumulated as weight[parent] + value).  Nodes are ordered by larger
// weight, then lower index; with values <= 0 a child never precedes its
// parent, so the first bs nodes of the order form a subtree that contains
// the root -- the most probable subgraph of size bs.
//
// Data layout: structure-of-arrays over node indices (children are appended
// after their parents, so index order is topological), a max-heap of the
// open (unexpanded, unselected) nodes keyed by (weight, -index) for the
// expansion step (O(w log s) per step), and per-node tree-cache rows: the
// root's keys and values are the last prefix row of the draft cache, every
// other expanded node owns one row, in the order the nodes were selected.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <utility>
#include <vector>

#include "../../include/swiftspec.h"

struct swiftspec_draft_tree {
  int32_t capacity = 0;
  std::vector<int32_t> token, parent, row, first_child, next_sibling;
  std::vector<double> weight;
  std::vector<uint8_t> expanded, selected;
  std::vector<int32_t> heap;  // open nodes, max-heap under `before`
  int32_t n_rows = 0, n_selected = 0;

  // a precedes b in the expansion / selection order
  bool before(int32_t a, int32_t b) const { return weight[a] > weight[b] || (weight[a] == weight[b] && a < b); }
  int32_t size() const { return (int32_t)token.size(); }

  void heap_push(int32_t v) {
    heap.push_back(v);
    std::push_heap(heap.begin(), heap.end(), [this](int32_t a, int32_t b) { return before(b, a); });
  }
  int32_t heap_pop() {
    std::pop_heap(heap.begin(), heap.end(), [this](int32_t a, int32_t b) { return before(b, a); });
    const int32_t v = heap.back();
    heap.pop_back();
    return v;
  }
  void rebuild_heap() {
    heap.clear();
    for (int32_t v = 0; v < size(); ++v)
      if (!expanded[v] && !selected[v]) heap.push_back(v);
    std::make_heap(heap.begin(), heap.end(), [this](int32_t a, int32_t b) { return before(b, a); });
  }
  int32_t add(int32_t tok, int32_t par, double w) {
    const int32_t v = size();
    token.push_back(tok);
    parent.push_back(par);
    row.push_back(-1);
    first_child.push_back(-1);
    next_sibling.push_back(-1);
    weight.push_back(w);
    expanded.push_back(0);
    selected.push_back(0);
    if (par >= 0) {  // keep children in index order: append at the end of the list
      int32_t* link = &first_child[par];
      while (*link >= 0) link = &next_sibling[*link];
      *link = v;
    }
    return v;
  }
  void reset(int32_t root_token) {
    token.clear();
    parent.clear();
    row.clear();
    first_child.clear();
    next_sibling.clear();
    weight.clear();
    expanded.clear();
    selected.clear();
    n_rows = n_selected = 0;
    add(root_token, -1, 0.0);
    rebuild_heap();
  }
  int32_t parent_row(int32_t v) const { return parent[v] <= 0 ? -1 : row[parent[v]]; }
};

// Host allocation failures inside the entry points surface as
// SWIFTSPEC_CAPACITY; no exception crosses the C ABI.
#define SS_NOTHROW_BEGIN try {
#define SS_NOTHROW_END \
  }                    \
  catch (...) {        \
    return SWIFTSPEC_CAPACITY; \
  }

extern "C" {

int swiftspec_draft_tree_create(int32_t capacity, int32_t root_token, swiftspec_draft_tree** out) {
  if (!out || capacity < 1) return SWIFTSPEC_INVALID_ARG;
  *out = nullptr;
  swiftspec_draft_tree* t = nullptr;
  SS_NOTHROW_BEGIN
  t = new swiftspec_draft_tree;
  t->capacity = capacity;
  t->token.reserve(capacity);
  t->reset(root_token);
  SS_NOTHROW_END
  *out = t;
  return SWIFTSPEC_OK;
}

void swiftspec_draft_tree_destroy(swiftspec_draft_tree* t) { delete t; }

int32_t swiftspec_draft_tree_size(const swiftspec_draft_tree* t) { return t ? t->size() : -1; }

int32_t swiftspec_draft_tree_rows(const swiftspec_draft_tree* t) { return t ? t->n_rows : -1; }

int swiftspec_draft_tree_nodes(const swiftspec_draft_tree* t, int32_t* token, int32_t* parent, double* weight,
                               int32_t* row, int32_t* expanded) {
  if (!t) return SWIFTSPEC_INVALID_ARG;
  for (int32_t v = 0; v < t->size(); ++v) {
    if (token) token[v] = t->token[v];
    if (parent) parent[v] = t->parent[v];
    if (weight) weight[v] = t->weight[v];
    if (row) row[v] = t->row[v];
    if (expanded) expanded[v] = t->expanded[v];
  }
  return SWIFTSPEC_OK;
}

int swiftspec_draft_tree_forest(const swiftspec_draft_tree* t, int32_t* parent_row) {
  if (!t || (!parent_row && t->n_rows > 0)) return SWIFTSPEC_INVALID_ARG;
  for (int32_t v = 1; v < t->size(); ++v)
    if (t->row[v] >= 0) parent_row[t->row[v]] = t->parent_row(v);
  return SWIFTSPEC_OK;
}

int swiftspec_draft_tree_select_leaves(swiftspec_draft_tree* t, int32_t w, int32_t* leaves, int32_t* parent_row,
                                       int32_t* n) {
  if (!t || !leaves || !parent_row || !n || w < 0) return SWIFTSPEC_INVALID_ARG;
  int32_t c = 0;
  while (c < w && !t->heap.empty()) {
    const int32_t v = t->heap_pop();
    t->selected[v] = 1;
    ++t->n_selected;
    if (v != 0) t->row[v] = t->n_rows++;
    leaves[c] = v;
    parent_row[c] = t->parent_row(v);
    ++c;
  }
  *n = c;
  return SWIFTSPEC_OK;
}

int swiftspec_draft_tree_expand(swiftspec_draft_tree* t, int32_t n, const int32_t* leaves, int32_t k,
                                const int32_t* tokens, const float* logprobs) {
  if (!t || n < 0 || k < 0 || (n > 0 && (!leaves || (k > 0 && (!tokens || !logprobs)))))
    return SWIFTSPEC_INVALID_ARG;
  // validate everything before changing anything
  for (int32_t j = 0; j < n; ++j) {
    const int32_t v = leaves[j];
    if (v < 0 || v >= t->size() || !t->selected[v] || t->expanded[v]) return SWIFTSPEC_INVALID_ARG;
    for (int32_t q = 0; q < j; ++q)
      if (leaves[q] == v) return SWIFTSPEC_INVALID_ARG;
    for (int32_t c = 0; c < k; ++c) {
      const float lp = logprobs[(size_t)j * k + c];
      if (!(lp <= 0.0f)) return SWIFTSPEC_INVALID_ARG;  // also rejects NaN
    }
  }
  if ((int64_t)t->size() + (int64_t)n * k > t->capacity) return SWIFTSPEC_CAPACITY;
  SS_NOTHROW_BEGIN
  // make room first, so that the appends below cannot fail half-way
  const size_t need = (size_t)t->size() + (size_t)n * k;
  for (auto* v : {&t->token, &t->parent, &t->row, &t->first_child, &t->next_sibling}) v->reserve(need);
  t->weight.reserve(need);
  t->expanded.reserve(need);
  t->selected.reserve(need);
  t->heap.reserve(t->heap.size() + (size_t)n * k);
  SS_NOTHROW_END
  for (int32_t j = 0; j < n; ++j) {
    const int32_t v = leaves[j];
    for (int32_t c = 0; c < k; ++c) {
      const int32_t ch =
          t->add(tokens[(size_t)j * k + c], v, t->weight[v] + (double)logprobs[(size_t)j * k + c]);
      t->heap_push(ch);
    }
    t->expanded[v] = 1;
    t->selected[v] = 0;
    --t->n_selected;
  }
  return SWIFTSPEC_OK;
}

int swiftspec_draft_tree_select_subgraph(const swiftspec_draft_tree* t, int32_t bs, int32_t* nodes,
                                         int32_t* parent, int32_t* tokens, int32_t* n) {
  if (!t || bs < 1 || !nodes || !parent || !n) return SWIFTSPEC_INVALID_ARG;
  const int32_t s = t->size(), m = bs < s ? bs : s;
  SS_NOTHROW_BEGIN
  std::vector<int32_t> all(s);
  for (int32_t v = 0; v < s; ++v) all[v] = v;
  std::nth_element(all.begin(), all.begin() + (m - 1), all.end(),
                   [t](int32_t a, int32_t b) { return t->before(a, b); });
  std::sort(all.begin(), all.begin() + m);  // by node index: parents first
  std::vector<int32_t> pos(s, -1);
  for (int32_t j = 0; j < m; ++j) pos[all[j]] = j;
  for (int32_t j = 0; j < m; ++j) {
    const int32_t v = all[j];
    nodes[j] = v;
    parent[j] = v == 0 ? -1 : pos[t->parent[v]];
    if (tokens) tokens[j] = t->token[v];
  }
  SS_NOTHROW_END
  *n = m;
  return SWIFTSPEC_OK;
}

int swiftspec_draft_tree_reroot(swiftspec_draft_tree* t, const int32_t* verified, int32_t n_verified,
                                int32_t* last, int32_t* path_rows, int32_t* keep, int32_t* pending,
                                int32_t* n_pending) {
  if (!t || !verified || n_verified < 2 || !last || !path_rows || !keep || !pending || !n_pending)
    return SWIFTSPEC_INVALID_ARG;
  if (verified[0] != t->token[0] || t->n_selected != 0) return SWIFTSPEC_INVALID_ARG;
  // walk: to the child carrying the next verified token while there is one
  int32_t end = 0, walked = 1, rows = 0, last_row = -1;
  for (; walked < n_verified; ++walked) {
    int32_t c = t->first_child[end];
    while (c >= 0 && t->token[c] != verified[walked]) c = t->next_sibling[c];
    if (c < 0) break;
    end = c;
    if (t->row[c] >= 0) {
      ++rows;
      last_row = t->row[c];
    }
  }
  if (walked < n_verified - 1) return SWIFTSPEC_INVALID_ARG;  // only the last token may be new
  *last = last_row;
  *path_rows = rows;
  if (walked == n_verified && end != 0 && t->expanded[end]) {
    SS_NOTHROW_BEGIN
    // keep end's subtree: nodes in index order, rows in row order
    const int32_t s = t->size();
    std::vector<int32_t> map(s, -1), sub;
    map[end] = 0;
    sub.push_back(end);
    for (int32_t v = end + 1; v < s; ++v)
      if (t->parent[v] >= 0 && map[t->parent[v]] >= 0) {
        map[v] = (int32_t)sub.size();
        sub.push_back(v);
      }
    std::vector<int32_t> kept_rows;
    for (int32_t v : sub)
      if (v != end && t->row[v] >= 0) kept_rows.push_back(t->row[v]);
    std::sort(kept_rows.begin(), kept_rows.end());
    std::vector<int32_t> rowmap(t->n_rows, -1);
    for (size_t j = 0; j < kept_rows.size(); ++j) rowmap[kept_rows[j]] = (int32_t)j;
    // built aside and swapped in, so that a failed allocation leaves the tree as it was
    swiftspec_draft_tree nt;
    nt.capacity = t->capacity;
    nt.token.reserve(t->capacity);
    const double base = t->weight[end];
    for (int32_t v : sub) {
      const int32_t nv = nt.add(t->token[v], v == end ? -1 : map[t->parent[v]], t->weight[v] - base);
      nt.expanded[nv] = t->expanded[v];
      nt.row[nv] = (v == end || t->row[v] < 0) ? -1 : rowmap[t->row[v]];
    }
    nt.n_rows = (int32_t)kept_rows.size();
    nt.n_selected = 0;
    nt.rebuild_heap();
    std::swap(*t, nt);
    SS_NOTHROW_END
    *keep = 1;
    *n_pending = 0;
    return SWIFTSPEC_OK;
  }
  // restart from the last verified token; the draft still lacks the keys
  // and values of the root (if never expanded) and of the verified tokens
  // after the walked expanded nodes
  int32_t np = 0;
  if (!t->expanded[0]) pending[np++] = t->token[0];
  for (int32_t j = 1 + rows; j < n_verified; ++j) pending[np++] = verified[j];
  SS_NOTHROW_BEGIN
  swiftspec_draft_tree nt;
  nt.capacity = t->capacity;
  nt.token.reserve(t->capacity);
  nt.reset(verified[n_verified - 1]);
  std::swap(*t, nt);
  SS_NOTHROW_END
  *n_pending = np;
  *keep = 0;
  return SWIFTSPEC_OK;
}

}  // extern "C"
