"""Pins of the budget / tree-construction oracle (oracle.budget) against what
the paper prints (R1-R4 of its worked numbers) and against brute force."""

import itertools

import numpy as np
import pytest

from oracle import budget as ob
from paper_2506_01986_amd import synth

MiB = 1 << 20


def test_r1_buffer_model_reproduces_the_paper_numbers():
    # Sec. 4: the Medusa 64-node mask takes 55 MB of buffers per query, the
    # SpecMemo "1-10-16-17" mask (44 nodes, 3 levels) 19.5 MB; over 20 queries
    # 390 MB and 1.1 GB; a 65% reduction.  Eq. 3 x 2 bytes, vocab 32000, in MiB.
    medusa = ob.buffer_bytes(1, 64, 42, 4, 32000, 2)
    assert medusa == 57_856_000 and round(medusa / MiB, 2) == 55.18
    # the 44-node mask's leaf count is not printed: 19.5 MB holds for S = 23 only
    fits = [s for s in range(1, 44) if round(ob.buffer_bytes(1, 44, s, 3, 32000, 2) / MiB, 1) == 19.5]
    assert fits == [23]
    small = ob.buffer_bytes(1, 44, 23, 3, 32000, 2)
    assert round(small / MiB, 2) == 19.53
    assert round(20 * small / MiB) == 391 and round(20 * medusa / (1 << 30), 1) == 1.1
    assert round(100 * (1 - small / medusa)) == 65


def test_r2_kv_model_with_head_dim():
    # Vicuna-7B: 32 layers, 32 KV heads, d = 128, fp16 -> 0.5 MiB per token, so
    # the 1 / 5 / 7 GB preallocations of Fig. 4 hold 2048 / 10240 / 14336 tokens.
    per_token = ob.kv_bytes(32, 1, 32, 128, 1, 2)
    assert per_token == MiB // 2
    assert [g * (1 << 30) // per_token for g in (1, 5, 7)] == [2048, 10240, 14336]
    # linear in every factor
    assert ob.kv_bytes(80, 3, 8, 128, 700, 2) == 3 * 700 * ob.kv_bytes(80, 1, 8, 128, 1, 2)


def test_r3_full_tree_closed_form():
    assert [ob.full_tree_nodes(10, l) for l in range(1, 5)] == [11, 111, 1111, 11111]
    assert [ob.full_tree_nodes(5, l) for l in range(1, 5)] == [6, 31, 156, 781]
    for k in range(1, 5):
        for l in range(0, 4):   # count the rank paths of length <= l directly
            count = sum(1 for n in range(l + 1) for _ in itertools.product(range(k), repeat=n))
            assert ob.full_tree_nodes(k, l) == count


def test_r4_default_tree_depth_profile():
    # Table 1, Medusa row: (leaves / nodes) of the 64-node tree cut after 1..4 levels
    t = synth.t64()
    prof = [ob.features(ob.truncate_depth(t.parent, t.depth, t.rank, l)[0]) for l in range(1, 5)]
    assert prof == [(11, 10), (34, 25), (57, 39), (64, 42)]


def _achievable(max_nodes, max_depth, arity):
    """Every (nodes, leaves) of an ordered tree with depth <= max_depth, at most
    `arity` children per node and at most max_nodes nodes (brute force over the
    BFS child-count sequences)."""
    found = set()
    # explicit stack of (node depths in BFS order, child counts chosen so far)
    stack = [([0], [])]
    while stack:
        depths, counts = stack.pop()
        i = len(counts)
        if i == len(depths):
            found.add((len(depths), sum(1 for c in counts if c == 0)))
            continue
        top = arity if depths[i] < max_depth else 0
        for c in range(top + 1):
            if len(depths) + c <= max_nodes:
                stack.append((depths + [depths[i] + 1] * c, counts + [c]))
    return found


@pytest.mark.parametrize("max_depth,arity", [(1, 1), (1, 3), (2, 1), (2, 2), (2, 3), (2, 5), (3, 2), (3, 3), (3, 4), (4, 2), (4, 3), (4, 4), (5, 2)])
def test_builder_feasibility_matches_brute_force(max_depth, arity):
    N = 12
    ok = _achievable(N, max_depth, arity)
    for nodes in range(1, N + 1):
        for leaves in range(1, N + 1):
            t = ob.build_tree(nodes, leaves, max_depth, arity)
            assert (t is not None) == ((nodes, leaves) in ok), (nodes, leaves)
            if t is None:
                continue
            parent, depth, rank = t
            assert ob.features(parent) == (nodes, leaves)
            assert max(depth) <= max_depth
            kids = {}
            for n in range(1, nodes):
                assert parent[n] < n and depth[n] == depth[parent[n]] + 1
                kids.setdefault(parent[n], []).append(rank[n])
            for p, r in kids.items():
                assert r == list(range(len(r))) and len(r) <= arity
            assert sum(1 for d in depth if d == 1) == min(arity, leaves, nodes - 1)


def test_builder_table1_custom_features():
    # The 44-node, 37-leaf custom tree of Table 1 (4 heads, top-10) and the
    # 64-node default's features are buildable exactly; the 3-level 44-node
    # mask with 23 leaves (R1) too.
    for nodes, leaves, levels in [(44, 37, 4), (64, 42, 4), (44, 23, 3), (11, 10, 1)]:
        p, d, r = ob.build_tree(nodes, leaves, levels, 10)
        assert ob.features(p) == (nodes, leaves) and max(d) <= levels
    # a tree cannot have as many leaves as nodes (Table 1's garbled 19/18, 28/27)
    assert ob.build_tree(18, 19, 2, 10) is None and ob.build_tree(27, 28, 3, 10) is None


def test_pruning_right_to_left():
    rng = np.random.default_rng(0)
    for _ in range(200):
        t = synth.random_tree(rng, int(rng.integers(1, 60)), max_depth=4, max_kids=5)
        keep = [int(x) for x in rng.integers(0, 12, size=4)]
        p, d, r = ob.prune_levels(t.parent, t.depth, t.rank, keep)
        paths = set(ob.to_paths(p, r))
        src = ob.to_paths(t.parent, t.rank)
        assert all(q[:-1] in paths for q in paths if q)                 # closed under parents
        for lev in range(1, 5):                                         # the leftmost candidates
            cand = [src[n] for n in range(t.n) if t.depth[n] == lev and src[t.parent[n]] in paths]
            want = cand[:keep[lev - 1]]
            assert sorted(q for q in paths if len(q) == lev) == sorted(want)
        n = int(rng.integers(1, t.n + 1))
        p2, d2, r2 = ob.prune_to(t.parent, t.depth, t.rank, n)
        assert len(p2) == n and all(p2[c] < c for c in range(1, n))


def _model():
    # a 7B-class model: 32 layers, 32 KV heads x 128, vocab 32000, fp16, heads of 0.6 GB
    return dict(base_model_bytes=13_476_839_424, head_bytes=600_000_000, layers=32, n_kv=32, head_dim=128,
                vocab=32000, elem_bytes=2, batch=1, query_count=20, query_length=128, default_heads=4)


def test_budget_plan_boundaries():
    t = synth.t64()
    tree = (list(t.parent), list(t.depth), list(t.rank))
    m = _model()
    cache = ob.kv_bytes(32, 1, 32, 128, 20 * 128, 2)
    assert cache == 2560 * MiB // 2
    full = m["base_model_bytes"] + 4 * m["head_bytes"] + cache + ob.buffer_bytes(1, 64, 42, 4, 32000, 2)
    plan = ob.plan_budget(full, default_tree=tree, **m)
    assert (plan["kind"], plan["heads"], plan["nodes"], plan["leaves"]) == (0, 4, 64, 42)
    assert plan["total_bytes"] == full
    # one byte short: the largest right-to-left pruning of the default tree, 63 nodes
    plan = ob.plan_budget(full - 1, default_tree=tree, **m)
    assert (plan["kind"], plan["heads"], plan["nodes"]) == (1, 4, 63)
    # heads no longer fit with any tree: one head fewer, the tree cut to 3 levels
    tight = m["base_model_bytes"] + 3 * m["head_bytes"] + cache + ob.buffer_bytes(1, 57, 39, 3, 32000, 2)
    plan = ob.plan_budget(tight, default_tree=tree, **m)
    assert (plan["kind"], plan["heads"], plan["nodes"], plan["leaves"]) == (2, 3, 57, 39)
    # nothing fits two heads and a 2-node tree
    floor = m["base_model_bytes"] + 2 * m["head_bytes"] + cache + ob.buffer_bytes(1, 2, 1, 2, 32000, 2)
    assert ob.plan_budget(floor, default_tree=tree, **m)["heads"] == 2
    assert ob.plan_budget(floor - 1, default_tree=tree, **m)["kind"] == -1
    # more memory never gives fewer heads or a smaller tree
    last = (0, 0)
    for mem in range(floor - 10, full + 10, (full - floor) // 97):
        p = ob.plan_budget(mem, default_tree=tree, **m)
        cur = (p["heads"], p["nodes"])
        assert cur >= last
        last = cur


def test_tree_sizes_from_slab_capacity():
    assert ob.plan_tree_sizes([10, 100, 50, 7], [80, 120, 50, 6], 64) == [64, 20, 0, 0]
