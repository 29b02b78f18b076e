"""Memory budget and tree construction of SpecMemo.  TEST INFRASTRUCTURE.

Plain Python over integers: the memory model of Sec. 3.1 (Eq. 1-6), the full
tree of Eq. 2, tree construction (Sec. 3.2: pruning right to left, building
from (nodes, leaves) features) and the budget search of Alg. 1 without its
quantisation step.  Only the tests may import this module; it shares nothing
with the library.

Trees are lists (parent, depth, rank) in BFS order: parent[0] = -1, every
parent precedes its children, siblings are ordered by rank and their ranks are
0, 1, 2, ...  A rank path is the tuple of ranks from the root to a node.

Readings where the paper is silent or garbled:
- Eq. 1's product omits the per-head dimension d that its legend defines; d is
  restored.  Eq. 6 multiplies the KV term by the precision again; the
  precision is applied once, inside each term.
- Eq. 3's l is the number of heads (the paper equates it with the tree's
  levels).
- Building from (nodes, leaves): the paper names the step but gives no method.
  Level 1 takes all k tokens of the first head when the leaf count allows
  (Sec. 3.2 keeps them all); the remaining internal nodes are made from leaves
  in breadth-first order (shallowest, then leftmost: the leftmost candidates
  carry the most probable tokens), the first ones taking the most children.
  That yields masks wide at the top, like the paper's.  The features are
  pinned (exact, and feasible whenever a tree with them exists); the shape
  itself is a reading (parity unpinned).
- Pruning right to left: at each level the rightmost nodes go first.  Pruning
  to n nodes keeps the first n nodes in BFS order, i.e. removes the deepest
  level's rightmost node first.
- Alg. 1 without quantisation: the default tree with the default heads if it
  fits; else, for the default heads and then one head fewer at a time down to
  two, the default tree cut to that depth and pruned node by node, the first
  (largest) that fits.
"""

from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple


# ---- Sec. 3.1: memory model -------------------------------------------------

def kv_bytes(layers: int, batch: int, n_kv: int, head_dim: int, tokens: int, elem_bytes: int) -> int:
    """Eq. 1 (with d): K and V for `tokens` positions of every layer and KV head."""
    return 2 * layers * batch * n_kv * head_dim * tokens * elem_bytes


def full_tree_nodes(arity: int, levels: int) -> int:
    """Eq. 2: nodes of the full arity-k tree with l levels below the root."""
    total, width = 0, 1
    for _ in range(levels + 1):
        total += width
        width *= arity
    return total


def buffer_bytes(batch: int, nodes: int, seqs: int, levels: int, vocab: int, elem_bytes: int) -> int:
    """Eq. 3 times the precision: node logits, candidate retrieval, acceptance lengths."""
    elems = batch * nodes * vocab + batch * seqs * levels * vocab + batch * seqs * levels * levels * vocab
    return elems * elem_bytes


def total_bytes(base_model_bytes: int, head_bytes: int, heads: int, kv: int, buffers: int) -> int:
    """Eq. 4-6: base model + heads + KV cache + runtime buffers."""
    return base_model_bytes + head_bytes * heads + kv + buffers


# ---- trees ------------------------------------------------------------------

def from_paths(paths: Sequence[Tuple[int, ...]]) -> Tuple[List[int], List[int], List[int]]:
    """BFS arrays of a set of rank paths (closed under prefixes)."""
    order = sorted(paths, key=lambda p: (len(p), p))
    index = {p: i for i, p in enumerate(order)}
    parent = [-1 if len(p) == 0 else index[p[:-1]] for p in order]
    depth = [len(p) for p in order]
    rank = [0 if len(p) == 0 else p[-1] for p in order]
    return parent, depth, rank


def to_paths(parent: Sequence[int], rank: Sequence[int]) -> List[Tuple[int, ...]]:
    paths: List[Tuple[int, ...]] = []
    for n in range(len(parent)):
        paths.append(() if parent[n] < 0 else paths[parent[n]] + (rank[n],))
    return paths


def features(parent: Sequence[int]) -> Tuple[int, int]:
    """(nodes, leaves): leaves are the candidate sequences of the mask."""
    n = len(parent)
    has_child = [False] * n
    for c in range(1, n):
        has_child[parent[c]] = True
    return n, sum(1 for x in has_child if not x)


def level_sizes(depth: Sequence[int]) -> List[int]:
    sizes = [0] * (max(depth) + 1)
    for d in depth:
        sizes[d] += 1
    return sizes


def build_tree(nodes: int, leaves: int, max_depth: int, arity: int) -> Optional[Tuple[List[int], List[int], List[int]]]:
    """A tree with exactly `nodes` nodes and `leaves` leaves, depth <= max_depth,
    at most `arity` children per node; None if the greedy finds none."""
    if nodes < 1 or leaves < 1 or max_depth < 0 or arity < 1:
        return None
    if nodes == 1:
        return ([-1], [0], [0]) if leaves == 1 else None
    if max_depth < 1:
        return None
    first = min(arity, leaves, nodes - 1)      # children of the root
    internal = nodes - 1 - leaves              # internal nodes besides the root
    rest = nodes - 1 - first                   # nodes below level 1
    if internal < 0 or rest < internal or rest > internal * arity:
        return None
    counts = []                                # children of each later internal node
    extra = rest - internal
    for _ in range(internal):
        x = min(arity - 1, extra)
        counts.append(1 + x)
        extra -= x
    paths = [()] + [(r,) for r in range(first)]
    kids: Dict[Tuple[int, ...], int] = {(): first}
    for c in counts:
        target = None
        for p in sorted(paths, key=lambda q: (len(q), q)):   # breadth-first: shallowest, then leftmost
            if len(p) < max_depth and kids.get(p, 0) == 0:
                target = p
                break
        if target is None:
            return None
        kids[target] = c
        paths += [target + (r,) for r in range(c)]
    return from_paths(paths)


def prune_levels(parent: Sequence[int], depth: Sequence[int], rank: Sequence[int],
                 keep: Sequence[int]) -> Tuple[List[int], List[int], List[int]]:
    """Right-to-left pruning: at depth d >= 1 keep at most keep[d-1] nodes, the
    leftmost whose parents are kept (levels past len(keep) keep nothing)."""
    kept = [False] * len(parent)
    kept[0] = True
    for d in range(1, max(depth) + 1):
        budget = keep[d - 1] if d - 1 < len(keep) else 0
        for n in range(len(parent)):
            if depth[n] == d and kept[parent[n]] and budget > 0:
                kept[n] = True
                budget -= 1
    paths = to_paths(parent, rank)
    return from_paths([paths[n] for n in range(len(parent)) if kept[n]])


def prune_to(parent: Sequence[int], depth: Sequence[int], rank: Sequence[int], n: int):
    """Right-to-left pruning to n nodes: the deepest level's rightmost node goes first."""
    n = max(1, min(n, len(parent)))
    return list(parent[:n]), list(depth[:n]), list(rank[:n])


def truncate_depth(parent, depth, rank, levels: int):
    """Keep the nodes of depth <= levels."""
    return prune_levels(parent, depth, rank, [len(parent)] * levels)


# ---- Alg. 1 without quantisation ------------------------------------------

def plan_budget(max_memory: int, base_model_bytes: int, head_bytes: int, layers: int, n_kv: int,
                head_dim: int, vocab: int, elem_bytes: int, batch: int, query_count: int,
                query_length: int, default_heads: int, default_tree) -> Dict[str, int]:
    """Heads and (nodes, leaves) of the mask that fit `max_memory`.

    kind: 0 the default tree and heads fit, 1 a pruned tree with the default
    heads, 2 fewer heads (at least 2), -1 nothing fits (Alg. 1 would quantise
    the base model next).
    """
    parent, depth, rank = default_tree
    cache = kv_bytes(layers, batch, n_kv, head_dim, query_count * query_length, elem_bytes)

    def need(h: int, nodes: int, leaves: int) -> int:
        return total_bytes(base_model_bytes, head_bytes, h,
                           cache, buffer_bytes(batch, nodes, leaves, h, vocab, elem_bytes))

    n0, s0 = features(parent)
    if need(default_heads, n0, s0) <= max_memory:
        return dict(kind=0, heads=default_heads, nodes=n0, leaves=s0, kv_bytes=cache,
                    total_bytes=need(default_heads, n0, s0))
    for h in range(default_heads, 1, -1):
        tp, td, tr = truncate_depth(parent, depth, rank, h)
        for n in range(len(tp), 1, -1):
            nodes, leaves = features(tp[:n])
            if need(h, nodes, leaves) <= max_memory:
                return dict(kind=1 if h == default_heads else 2, heads=h, nodes=nodes, leaves=leaves,
                            kv_bytes=cache, total_bytes=need(h, nodes, leaves))
    return dict(kind=-1, heads=0, nodes=0, leaves=0, kv_bytes=cache, total_bytes=0)


def plan_tree_sizes(seq_len: Sequence[int], seq_cap: Sequence[int], default_nodes: int) -> List[int]:
    """Per sequence, the tree nodes its slab can hold this step: the default
    tree's size, capped by the slab's free rows (0: no room for a tree)."""
    return [max(0, min(default_nodes, c - l)) for l, c in zip(seq_len, seq_cap)]
