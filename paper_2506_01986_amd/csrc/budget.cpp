// Host half of libspecmemo: SpecMemo's memory model (Sec. 3.1, Eq. 1-6), tree
// construction from (nodes, leaves) features and right-to-left pruning
// (Sec. 3.2), and the budget search of Alg. 1 without its quantisation step.
// Plain integer code over host arrays; no HIP call.
#include "specmemo.h"

#include <algorithm>
#include <vector>

#include "internal.h"

using namespace specmemo;

namespace {

constexpr int64_t kMaxBuildNodes = int64_t(1) << 24;   // bounds the builder's staging arrays

// Product of non-negative factors; -1 if it does not fit int64.
int64_t checked_product(std::initializer_list<int64_t> factors) {
  int64_t r = 1;
  for (int64_t f : factors)
    if (__builtin_mul_overflow(r, f, &r)) return -1;
  return r;
}

int64_t checked_sum(std::initializer_list<int64_t> terms) {
  int64_t r = 0;
  for (int64_t t : terms)
    if (__builtin_add_overflow(r, t, &r)) return -1;
  return r;
}

// Eq. 1 with d; -1 on overflow (arguments already checked non-negative).
int64_t kv_bytes(int64_t layers, int64_t batch, int64_t n_kv, int64_t head_dim, int64_t tokens, int64_t elem) {
  return checked_product({2, layers, batch, n_kv, head_dim, tokens, elem});
}

// Eq. 3 x precision; -1 on overflow.
int64_t buffer_bytes(int64_t b, int64_t nodes, int64_t seqs, int64_t levels, int64_t w, int64_t elem) {
  const int64_t logits = checked_product({b, nodes, w});           // node logits
  const int64_t retrieve = checked_product({b, seqs, levels, w});  // candidate retrieval
  const int64_t lengths = checked_product({b, seqs, levels, levels, w});  // acceptance lengths
  if (logits < 0 || retrieve < 0 || lengths < 0) return -1;
  const int64_t elems = checked_sum({logits, retrieve, lengths});
  return elems < 0 ? -1 : checked_product({elems, elem});
}

// Eq. 4-6; -1 on overflow.
int64_t total_bytes(int64_t base, int64_t head_bytes, int64_t heads, int64_t kv, int64_t buffers) {
  const int64_t h = checked_product({head_bytes, heads});
  return h < 0 ? -1 : checked_sum({base, h, kv, buffers});
}

// Breadth-first tree conventions of the header's memory-budget section.
int check_bfs_tree(int32_t n, const int32_t *parent, const int32_t *depth, const int32_t *rank, const char *what) {
  if (n < 1) return fail(SPECMEMO_E_ARG, "%s: n=%d, need at least the root", what, n);
  if (!parent || !depth || !rank) return fail(SPECMEMO_E_ARG, "%s: NULL tree array", what);
  if (parent[0] != -1 || depth[0] != 0 || rank[0] != 0)
    return fail(SPECMEMO_E_TREE, "%s: node 0 must be the root (parent -1, depth 0, rank 0)", what);
  for (int32_t i = 1; i < n; ++i) {
    const int32_t p = parent[i];
    if (p < 0 || p >= i) return fail(SPECMEMO_E_TREE, "%s: parent[%d]=%d is not an earlier node", what, i, p);
    if (depth[i] != depth[p] + 1)
      return fail(SPECMEMO_E_TREE, "%s: depth[%d]=%d, its parent's is %d", what, i, depth[i], depth[p]);
    if (rank[i] < 0) return fail(SPECMEMO_E_TREE, "%s: rank[%d]=%d is negative", what, i, rank[i]);
    if (i > 1) {
      const int32_t pd = depth[i - 1], pp = parent[i - 1], pr = rank[i - 1];
      const bool after = depth[i] != pd ? depth[i] > pd : p != pp ? p > pp : rank[i] > pr;
      if (!after)
        return fail(SPECMEMO_E_TREE, "%s: node %d is out of breadth-first order (depth, parent, rank)", what, i);
    }
  }
  return SPECMEMO_OK;
}

// Leaves of a valid breadth-first tree's first `n` nodes.
int32_t count_leaves(int32_t n, const int32_t *parent, std::vector<int32_t> *kids) {
  kids->assign(n, 0);
  for (int32_t i = 1; i < n; ++i) ++(*kids)[parent[i]];
  return int32_t(std::count(kids->begin(), kids->end(), 0));
}

}  // namespace

extern "C" {

int64_t specmemo_mem_kv_bytes(int32_t layers, int32_t batch, int32_t n_kv, int32_t head_dim, int64_t tokens,
                              int32_t elem_bytes) {
  if (layers < 0 || batch < 0 || n_kv < 0 || head_dim < 0 || tokens < 0 || elem_bytes < 1) {
    fail(SPECMEMO_E_ARG, "kv bytes: negative size or elem_bytes < 1");
    return -1;
  }
  const int64_t r = kv_bytes(layers, batch, n_kv, head_dim, tokens, elem_bytes);
  if (r < 0) fail(SPECMEMO_E_ARG, "kv bytes overflow int64");
  else ok();
  return r;
}

int64_t specmemo_mem_buffer_bytes(int32_t batch, int32_t nodes, int32_t seqs, int32_t levels, int32_t vocab,
                                  int32_t elem_bytes) {
  if (batch < 0 || nodes < 0 || seqs < 0 || levels < 0 || vocab < 0 || elem_bytes < 1) {
    fail(SPECMEMO_E_ARG, "buffer bytes: negative size or elem_bytes < 1");
    return -1;
  }
  const int64_t r = buffer_bytes(batch, nodes, seqs, levels, vocab, elem_bytes);
  if (r < 0) fail(SPECMEMO_E_ARG, "buffer bytes overflow int64");
  else ok();
  return r;
}

int64_t specmemo_mem_total_bytes(int64_t base_model_bytes, int64_t head_bytes, int32_t heads, int64_t kv,
                                 int64_t buffers) {
  if (base_model_bytes < 0 || head_bytes < 0 || heads < 0 || kv < 0 || buffers < 0) {
    fail(SPECMEMO_E_ARG, "total bytes: negative term");
    return -1;
  }
  const int64_t r = total_bytes(base_model_bytes, head_bytes, heads, kv, buffers);
  if (r < 0) fail(SPECMEMO_E_ARG, "total bytes overflow int64");
  else ok();
  return r;
}

int64_t specmemo_tree_full_nodes(int32_t arity, int32_t levels) {
  if (arity < 1 || levels < 0) {
    fail(SPECMEMO_E_ARG, "full tree: arity=%d levels=%d", arity, levels);
    return -1;
  }
  // Horner form of Eq. 2: 1 + k (1 + k (1 + ...)), one factor per level
  int64_t n = 1;
  for (int32_t i = 0; i < levels; ++i) {
    if (__builtin_mul_overflow(n, int64_t(arity), &n) || __builtin_add_overflow(n, int64_t(1), &n)) {
      fail(SPECMEMO_E_ARG, "full tree of arity %d and %d levels overflows int64", arity, levels);
      return -1;
    }
  }
  ok();
  return n;
}

int specmemo_tree_build(int32_t nodes, int32_t leaves, int32_t max_depth, int32_t arity, int32_t *parent,
                        int32_t *depth, int32_t *rank) {
  if (nodes < 1 || leaves < 1 || max_depth < 0 || arity < 1)
    return fail(SPECMEMO_E_ARG, "tree build: nodes=%d leaves=%d max_depth=%d arity=%d", nodes, leaves, max_depth,
                arity);
  if (nodes > kMaxBuildNodes) return fail(SPECMEMO_E_ARG, "tree build: nodes=%d exceeds %lld", nodes,
                                          static_cast<long long>(kMaxBuildNodes));
  if (!parent || !depth || !rank) return fail(SPECMEMO_E_ARG, "tree build: NULL output array");
  if (nodes == 1) {
    if (leaves != 1) return fail(SPECMEMO_E_TREE, "a 1-node tree has 1 leaf, not %d", leaves);
    parent[0] = -1, depth[0] = 0, rank[0] = 0;
    return ok();
  }
  if (max_depth < 1) return fail(SPECMEMO_E_TREE, "%d nodes do not fit depth 0", nodes);
  // Level 1 keeps as many of the first head's tokens as the leaf count allows.
  // Below it, `inner` internal nodes (all but the root) share the remaining
  // `below` nodes, each taking between 1 and `arity` children.
  const int64_t first = std::min<int64_t>({arity, leaves, nodes - 1});
  const int64_t inner = int64_t(nodes) - 1 - leaves;
  const int64_t below = int64_t(nodes) - 1 - first;
  if (inner < 0 || below < inner || below > inner * arity)
    return fail(SPECMEMO_E_TREE, "no tree has %d nodes and %d leaves with at most %d children per node", nodes,
                leaves, arity);
  std::vector<int32_t> P(nodes), D(nodes), R(nodes);
  P[0] = -1, D[0] = 0, R[0] = 0;
  int32_t made = 1;
  for (int32_t r = 0; r < first; ++r, ++made) P[made] = 0, D[made] = 1, R[made] = r;
  // Nodes are made in breadth-first order, so scanning them in order visits
  // the leaves shallowest first, then leftmost; each internal node takes one
  // child plus as many of the spare ones as arity allows.
  int64_t spare = below - inner;
  int32_t next = 1;
  for (int64_t j = 0; j < inner; ++j) {
    while (next < made && D[next] >= max_depth) ++next;
    if (next == made)
      return fail(SPECMEMO_E_TREE, "no tree has %d nodes and %d leaves within depth %d and arity %d", nodes,
                  leaves, max_depth, arity);
    const int64_t extra = std::min<int64_t>(arity - 1, spare);
    spare -= extra;
    for (int32_t r = 0; r <= extra; ++r, ++made) P[made] = next, D[made] = D[next] + 1, R[made] = r;
    ++next;
  }
  std::copy(P.begin(), P.end(), parent);
  std::copy(D.begin(), D.end(), depth);
  std::copy(R.begin(), R.end(), rank);
  return ok();
}

int32_t specmemo_tree_leaves(int32_t n, const int32_t *parent, const int32_t *depth, const int32_t *rank) {
  if (check_bfs_tree(n, parent, depth, rank, "tree leaves")) return -1;
  std::vector<int32_t> kids;
  const int32_t s = count_leaves(n, parent, &kids);
  ok();
  return s;
}

int specmemo_tree_prune(int32_t n, const int32_t *parent, const int32_t *depth, const int32_t *rank,
                        int32_t n_keep, const int32_t *keep, int32_t *n_out, int32_t *parent_out,
                        int32_t *depth_out, int32_t *rank_out) {
  int rc;
  if ((rc = check_bfs_tree(n, parent, depth, rank, "tree prune"))) return rc;
  if (n_keep < 0 || (n_keep > 0 && !keep)) return fail(SPECMEMO_E_ARG, "tree prune: n_keep=%d", n_keep);
  if (!n_out || !parent_out || !depth_out || !rank_out) return fail(SPECMEMO_E_ARG, "tree prune: NULL output");
  std::vector<int32_t> left(keep, keep + n_keep);
  for (int32_t d = 0; d < n_keep; ++d)
    if (left[d] < 0) return fail(SPECMEMO_E_ARG, "tree prune: keep[%d]=%d is negative", d, left[d]);
  // One pass in breadth-first order: parents are decided before their
  // children, and each level's survivors are its leftmost eligible nodes.
  // Node i is written at slot m <= i after it has been read, so the outputs
  // may be the inputs themselves.
  std::vector<int32_t> new_id(n, -1);
  new_id[0] = 0;
  int32_t m = 1;
  parent_out[0] = -1, depth_out[0] = 0, rank_out[0] = 0;
  for (int32_t i = 1; i < n; ++i) {
    const int32_t p = new_id[parent[i]], d = depth[i], r = rank[i];
    if (p < 0 || d > n_keep || left[d - 1] == 0) continue;
    --left[d - 1];
    new_id[i] = m;
    parent_out[m] = p, depth_out[m] = d, rank_out[m] = r;
    ++m;
  }
  *n_out = m;
  return ok();
}

int specmemo_plan_budget(const specmemo_budget *mb, int32_t n, const int32_t *parent, const int32_t *depth,
                         const int32_t *rank, specmemo_budget_plan *out) {
  if (!mb || !out) return fail(SPECMEMO_E_ARG, "plan budget: NULL model or output");
  const specmemo_budget &m = *mb;
  if (m.max_memory < 0 || m.base_model_bytes < 0 || m.head_bytes < 0)
    return fail(SPECMEMO_E_ARG, "plan budget: negative byte count");
  if (m.layers < 1 || m.n_kv < 1 || m.head_dim < 1 || m.vocab < 1 || m.elem_bytes < 1 || m.batch < 1 ||
      m.query_count < 1 || m.query_length < 1)
    return fail(SPECMEMO_E_ARG, "plan budget: layers, n_kv, head_dim, vocab, elem_bytes, batch, query_count "
                                "and query_length must be positive");
  if (m.default_heads < 2) return fail(SPECMEMO_E_ARG, "plan budget: default_heads=%d < 2", m.default_heads);
  int rc;
  if ((rc = check_bfs_tree(n, parent, depth, rank, "plan budget"))) return rc;
  if (depth[n - 1] > m.default_heads)
    return fail(SPECMEMO_E_TREE, "plan budget: default tree depth %d exceeds default_heads=%d", depth[n - 1],
                m.default_heads);
  // ComputeMinCache: the KV cache of n queries of m tokens
  const int64_t cache = kv_bytes(m.layers, m.batch, m.n_kv, m.head_dim,
                                 int64_t(m.query_count) * m.query_length, m.elem_bytes);
  if (cache < 0) return fail(SPECMEMO_E_ARG, "plan budget: KV cache bytes overflow int64");
  // Eq. 6 of (heads, nodes, leaves); -1 (never fits) when it overflows
  auto need = [&](int32_t h, int32_t nodes, int32_t leaves) -> int64_t {
    const int64_t buf = buffer_bytes(m.batch, nodes, leaves, h, m.vocab, m.elem_bytes);
    return buf < 0 ? -1 : total_bytes(m.base_model_bytes, m.head_bytes, h, cache, buf);
  };
  auto fits = [&](int64_t t) { return t >= 0 && t <= m.max_memory; };
  auto plan = [&](int32_t kind, int32_t h, int32_t nodes, int32_t leaves, int64_t t) {
    out->kind = kind, out->heads = h, out->nodes = nodes, out->leaves = leaves;
    out->kv_bytes = cache, out->total_bytes = t;
    return ok();
  };
  std::vector<int32_t> kids;
  const int32_t leaves0 = count_leaves(n, parent, &kids);
  if (fits(need(m.default_heads, n, leaves0)))
    return plan(SPECMEMO_PLAN_DEFAULT, m.default_heads, n, leaves0, need(m.default_heads, n, leaves0));
  // ExploreTree, then one head fewer at a time.  Cutting a breadth-first tree
  // to depth h keeps a prefix, and pruning it right to left one node at a
  // time drops its last node: that node is a leaf, and its parent becomes
  // one when it loses its only remaining child.
  for (int32_t h = m.default_heads; h >= 2; --h) {
    const int32_t len = int32_t(std::upper_bound(depth, depth + n, h) - depth);
    int32_t leaves = count_leaves(len, parent, &kids);
    for (int32_t cnt = len; cnt >= 2; --cnt) {
      const int64_t t = need(h, cnt, leaves);
      if (fits(t))
        return plan(h == m.default_heads ? SPECMEMO_PLAN_PRUNED : SPECMEMO_PLAN_FEWER_HEADS, h, cnt, leaves, t);
      if (--kids[parent[cnt - 1]] > 0) --leaves;
    }
  }
  return plan(SPECMEMO_PLAN_NONE, 0, 0, 0, 0);
}

int specmemo_plan_tree_sizes(int32_t B, const int32_t *seq_len_h, const int32_t *seq_cap_h, int32_t default_nodes,
                             int32_t *nodes_out) {
  if (B < 0) return fail(SPECMEMO_E_ARG, "tree sizes: B=%d", B);
  if (default_nodes < 1 || default_nodes > SPECMEMO_MAX_TREE_NODES)
    return fail(SPECMEMO_E_ARG, "tree sizes: default_nodes=%d outside 1..%d", default_nodes,
                SPECMEMO_MAX_TREE_NODES);
  if (B > 0 && (!seq_len_h || !seq_cap_h || !nodes_out)) return fail(SPECMEMO_E_ARG, "tree sizes: NULL array");
  for (int32_t b = 0; b < B; ++b)
    if (seq_len_h[b] < 0 || seq_cap_h[b] < 0)
      return fail(SPECMEMO_E_ARG, "tree sizes: seq_len[%d]=%d seq_cap[%d]=%d", b, seq_len_h[b], b, seq_cap_h[b]);
  for (int32_t b = 0; b < B; ++b) {
    const int64_t free_rows = int64_t(seq_cap_h[b]) - seq_len_h[b];
    nodes_out[b] = int32_t(std::max<int64_t>(0, std::min<int64_t>(default_nodes, free_rows)));
  }
  return ok();
}

}  // extern "C"
