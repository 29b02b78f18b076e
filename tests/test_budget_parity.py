"""Parity of the library's host budget and tree-construction calls with the
oracle (oracle.budget): bit-exact on every integer, on seeded random inputs
and exhaustively on small ones, plus their argument and tree checks.  These
calls make no HIP call, so the whole file runs without a GPU."""

import numpy as np
import pytest

from oracle import budget as ob
from paper_2506_01986_amd import specmemo as sm
from paper_2506_01986_amd import synth


def _tree(t):
    return (list(map(int, t.parent)), list(map(int, t.depth)), list(map(int, t.rank)))


def _same(a, b):
    assert [list(map(int, x)) for x in a] == [list(map(int, x)) for x in b]


def test_memory_model_matches_oracle():
    rng = np.random.default_rng(1)
    for _ in range(500):
        layers, batch, n_kv, d = (int(x) for x in rng.integers(0, [200, 64, 128, 512]))
        tokens, elem = int(rng.integers(0, 1 << 20)), int(rng.integers(1, 5))
        assert sm.mem_kv_bytes(layers, batch, n_kv, d, tokens, elem) == ob.kv_bytes(layers, batch, n_kv, d, tokens, elem)
        b, n, s, lv = (int(x) for x in rng.integers(0, [64, 1200, 1200, 16]))
        w = int(rng.integers(0, 260_000))
        assert sm.mem_buffer_bytes(b, n, s, lv, w, elem) == ob.buffer_bytes(b, n, s, lv, w, elem)
        base, head, heads = int(rng.integers(0, 1 << 40)), int(rng.integers(0, 1 << 32)), int(rng.integers(0, 16))
        kv, buf = int(rng.integers(0, 1 << 40)), int(rng.integers(0, 1 << 36))
        assert sm.mem_total_bytes(base, head, heads, kv, buf) == ob.total_bytes(base, head, heads, kv, buf)
    for k in range(1, 12):
        for lv in range(0, 9):
            assert sm.tree_full_nodes(k, lv) == ob.full_tree_nodes(k, lv)


def test_memory_model_overflow_and_bad_arguments():
    big = (1 << 31) - 1
    with pytest.raises(sm.SpecmemoError, match="overflow"):
        sm.mem_kv_bytes(big, big, big, big, 1 << 40, 2)
    with pytest.raises(sm.SpecmemoError, match="overflow"):
        sm.mem_buffer_bytes(big, big, big, big, big, 4)
    with pytest.raises(sm.SpecmemoError, match="overflow"):
        sm.mem_total_bytes((1 << 62), (1 << 62), 2, 0, 0)
    with pytest.raises(sm.SpecmemoError, match="overflow"):
        sm.tree_full_nodes(10, 19)
    assert sm.tree_full_nodes(10, 18) == ob.full_tree_nodes(10, 18)
    for bad in [(-1, 1, 1, 1, 1, 2), (1, 1, 1, 1, -1, 2), (1, 1, 1, 1, 1, 0)]:
        with pytest.raises(sm.SpecmemoError):
            sm.mem_kv_bytes(*bad)
    with pytest.raises(sm.SpecmemoError):
        sm.tree_full_nodes(0, 3)


@pytest.mark.parametrize("max_depth", [0, 1, 2, 3, 4, 6])
@pytest.mark.parametrize("arity", [1, 2, 3, 5, 10])
def test_builder_matches_oracle_exhaustively(max_depth, arity):
    for nodes in range(1, 41):
        for leaves in range(1, 42):
            want = ob.build_tree(nodes, leaves, max_depth, arity)
            if want is None:
                with pytest.raises(sm.SpecmemoError) as e:
                    sm.tree_build(nodes, leaves, max_depth, arity)
                assert e.value.name == "E_TREE"
            else:
                _same(sm.tree_build(nodes, leaves, max_depth, arity), want)


def test_builder_matches_oracle_on_large_trees():
    rng = np.random.default_rng(2)
    done = 0
    while done < 60:
        nodes = int(rng.integers(41, 400))
        leaves = int(rng.integers(1, nodes))
        depth, arity = int(rng.integers(1, 8)), int(rng.integers(1, 12))
        want = ob.build_tree(nodes, leaves, depth, arity)
        if want is None:
            with pytest.raises(sm.SpecmemoError):
                sm.tree_build(nodes, leaves, depth, arity)
            continue
        got = sm.tree_build(nodes, leaves, depth, arity)
        _same(got, want)
        assert sm.tree_leaves(*got) == leaves
        done += 1


def test_builder_arguments():
    for bad in [(0, 1, 3, 2), (5, 0, 3, 2), (5, 2, -1, 2), (5, 2, 3, 0), ((1 << 24) + 1, 5, 3, 2)]:
        with pytest.raises(sm.SpecmemoError) as e:
            sm.tree_build(*bad)
        assert e.value.name == "E_ARG"


def _random_keep(rng, levels):
    return [int(x) for x in rng.integers(0, 14, size=levels)]


def test_prune_matches_oracle():
    rng = np.random.default_rng(3)
    trees = [synth.t16(), synth.t64()] + [synth.random_tree(rng, int(rng.integers(1, 129)), max_depth=4, max_kids=10)
                                          for _ in range(300)]
    for t in trees:
        for levels in (0, 1, 3, 4, 6):
            keep = _random_keep(rng, levels)
            want = ob.prune_levels(*_tree(t), keep) if levels else ([-1], [0], [0])
            _same(sm.tree_prune(t.parent, t.depth, t.rank, keep), want)
        # cutting to depth h keeps every node of depth <= h
        for h in range(0, 5):
            want = ob.truncate_depth(*_tree(t), h) if h else ([-1], [0], [0])
            _same(sm.tree_prune(t.parent, t.depth, t.rank, [t.n] * h), want)


def test_prune_in_place():
    rng = np.random.default_rng(4)
    lib = sm.load()
    import ctypes as C
    for _ in range(50):
        t = synth.random_tree(rng, int(rng.integers(2, 129)), max_depth=4, max_kids=10)
        keep = np.asarray(_random_keep(rng, 4), np.int32)
        p, d, r = (np.ascontiguousarray(a, dtype=np.int32).copy() for a in (t.parent, t.depth, t.rank))
        m = C.c_int32(0)
        rc = lib.specmemo_tree_prune(t.n, p.ctypes.data, d.ctypes.data, r.ctypes.data, 4, keep.ctypes.data,
                                     C.addressof(m), p.ctypes.data, d.ctypes.data, r.ctypes.data)
        assert rc == 0
        _same((p[:m.value], d[:m.value], r[:m.value]), ob.prune_levels(*_tree(t), list(keep)))


def test_tree_checks():
    t = synth.t16()
    base = [np.asarray(a, np.int32).copy() for a in (t.parent, t.depth, t.rank)]
    assert sm.tree_leaves(*base) == ob.features(list(t.parent))[1]
    cases = []
    p, d, r = (a.copy() for a in base); p[0] = 0; cases.append((p, d, r))        # no root
    p, d, r = (a.copy() for a in base); p[5] = 7; cases.append((p, d, r))        # parent after child
    p, d, r = (a.copy() for a in base); d[6] = 3; cases.append((p, d, r))        # depth off its parent's
    p, d, r = (a.copy() for a in base); r[2] = 0; cases.append((p, d, r))        # duplicate sibling rank
    p, d, r = (a.copy() for a in base); r[3], r[4] = r[4], r[3]; cases.append((p, d, r))   # siblings out of order
    p, d, r = (a.copy() for a in base); r[1] = -1; cases.append((p, d, r))       # negative rank
    for c in cases:
        with pytest.raises(sm.SpecmemoError) as e:
            sm.tree_leaves(*c)
        assert e.value.name == "E_TREE"
        with pytest.raises(sm.SpecmemoError) as e:
            sm.tree_prune(*c, [4, 4, 4])
        assert e.value.name == "E_TREE"
    with pytest.raises(sm.SpecmemoError) as e:
        sm.tree_prune(*base, [4, -1, 4])
    assert e.value.name == "E_ARG"


def _model(**over):
    m = dict(base_model_bytes=13_476_839_424, head_bytes=600_000_000, layers=32, n_kv=32, head_dim=128,
             vocab=32000, elem_bytes=2, batch=1, query_count=20, query_length=128, default_heads=4)
    m.update(over)
    return m


def _sweep(m, tree, count):
    heads = m["default_heads"]
    cache = ob.kv_bytes(m["layers"], m["batch"], m["n_kv"], m["head_dim"], m["query_count"] * m["query_length"],
                        m["elem_bytes"])
    lo = m["base_model_bytes"] + 2 * m["head_bytes"] + cache
    n, s = ob.features(tree[0])
    hi = m["base_model_bytes"] + heads * m["head_bytes"] + cache + \
        ob.buffer_bytes(m["batch"], n, s, heads, m["vocab"], m["elem_bytes"])
    mems = list(np.linspace(lo - 1000, hi + 1000, count).astype(np.int64)) + [lo - 1, lo, hi - 1, hi, 0]
    for mem in mems:
        want = ob.plan_budget(int(mem), default_tree=tree, **m)
        got = sm.plan_budget(int(mem), default_tree=tree, **m)
        assert got == want, (int(mem), got, want)


def test_plan_budget_matches_oracle_t64():
    _sweep(_model(), _tree(synth.t64()), 400)


def test_plan_budget_matches_oracle_random():
    rng = np.random.default_rng(5)
    for i in range(40):
        heads = int(rng.integers(2, 6))
        t = synth.random_tree(rng, int(rng.integers(2, min(129, ob.full_tree_nodes(10, heads) + 1))),
                              max_depth=heads, max_kids=10)
        m = _model(default_heads=heads, batch=int(rng.integers(1, 11)), layers=int(rng.integers(1, 81)),
                   n_kv=int(rng.integers(1, 65)), vocab=int(rng.integers(1000, 130_000)),
                   elem_bytes=int(rng.choice([1, 2, 4])), query_count=int(rng.integers(1, 50)),
                   query_length=int(rng.integers(1, 4096)), head_bytes=int(rng.integers(0, 2_000_000_000)))
        _sweep(m, _tree(t), 40)


def test_plan_budget_arguments():
    t = _tree(synth.t64())
    with pytest.raises(sm.SpecmemoError) as e:
        sm.plan_budget(1 << 40, default_tree=t, **_model(default_heads=1))
    assert e.value.name == "E_ARG"
    with pytest.raises(sm.SpecmemoError) as e:
        sm.plan_budget(1 << 40, default_tree=t, **_model(default_heads=3))    # T64 is 4 levels deep
    assert e.value.name == "E_TREE"
    with pytest.raises(sm.SpecmemoError) as e:
        sm.plan_budget(1 << 40, default_tree=t, **_model(vocab=0))
    assert e.value.name == "E_ARG"
    with pytest.raises(sm.SpecmemoError, match="overflow"):
        sm.plan_budget(1 << 40, default_tree=t, **_model(layers=(1 << 31) - 1, query_count=(1 << 31) - 1,
                                                         query_length=(1 << 31) - 1))


def test_tree_sizes_match_oracle():
    rng = np.random.default_rng(6)
    for _ in range(50):
        B = int(rng.integers(0, 40))
        ln = rng.integers(0, 5000, size=B)
        cap = ln + rng.integers(-200, 300, size=B)
        cap = np.maximum(cap, 0)
        dn = int(rng.integers(1, 129))
        assert list(sm.plan_tree_sizes(ln, cap, dn)) == ob.plan_tree_sizes(list(ln), list(cap), dn)
    with pytest.raises(sm.SpecmemoError):
        sm.plan_tree_sizes([1], [5], 129)
    with pytest.raises(sm.SpecmemoError):
        sm.plan_tree_sizes([-1], [5], 64)
