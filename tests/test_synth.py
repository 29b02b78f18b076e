"""Seeded synthetic inputs: determinism, tree fixtures, pool layout."""

import os

import numpy as np
import pytest

from paper_2506_01986_amd import configs, synth

HERE = os.path.dirname(os.path.abspath(__file__))


def _arrays(wl):
    return dict(lens=wl.lens, node_off=wl.node_off, parent=wl.parent, depth=wl.depth,
                rank=wl.rank, hidden=wl.hidden, head_w=wl.head_w, root_tok=wl.root_tok, q=wl.q,
                pool_k=wl.pool_k, pool_v=wl.pool_v, seq_base=wl.seq_base, seq_cap=wl.seq_cap,
                base_logits=wl.base_logits, p_accept=wl.p_accept)


def test_same_seed_same_bytes():
    a, b = synth.make(configs.TINY_FP32), synth.make(configs.TINY_FP32)
    for k, x in _arrays(a).items():
        assert np.array_equal(x.view(np.uint8), _arrays(b)[k].view(np.uint8)), k
    assert a.plan == b.plan and a.plan_path == b.plan_path


def test_other_seed_other_bytes():
    a, b = synth.make(configs.TINY_FP32), synth.make(configs.TINY_FP32, seed=99)
    assert not np.array_equal(a.q, b.q)


def test_chunked_draws_do_not_depend_on_threads(monkeypatch):
    ss = np.random.SeedSequence(7)
    n = 3 * synth.CHUNK + 123
    monkeypatch.setattr(synth, "_NTHREADS", 1)
    x1 = synth.normals(ss, n)
    monkeypatch.setattr(synth, "_NTHREADS", 8)
    x8 = synth.normals(np.random.SeedSequence(7), n)
    assert np.array_equal(x1, x8)


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1e-3], np.float32)
    b = synth.to_bf16_bits(x)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa (1.0) wins;
    # 1 + 3*2^-8 ties between 1+2^-7 and 1+2^-6: even is 1 + 2^-6.
    assert list(synth.bf16_bits_to_f32(b)[:4]) == [1.0, 1.0, 1.0 + 2 ** -6, -2.5]


def _levels(t):
    return np.bincount(t.depth).tolist()


def _leaves(t):
    has_kid = np.zeros(t.n, bool)
    has_kid[t.parent[1:]] = True
    return np.nonzero(~has_kid)[0]


def _check_tree(t, n_heads, topk):
    assert t.parent[0] == -1 and t.depth[0] == 0
    for n in range(1, t.n):
        p = t.parent[n]
        assert 0 <= p < n
        assert t.depth[n] == t.depth[p] + 1 <= n_heads
        assert 0 <= t.rank[n] < topk[t.depth[n] - 1]
    assert np.all(np.diff(t.depth) >= 0), "BFS order"
    for u in range(t.n):
        ranks = [int(t.rank[c]) for c in synth.children(t, u)]
        assert len(set(ranks)) == len(ranks), "sibling ranks distinct"


def test_t16():
    t = synth.t16()
    _check_tree(t, 3, (4, 2, 2))
    assert _levels(t) == [1, 4, 6, 5]
    assert _leaves(t).tolist() == [8, 10, 11, 12, 13, 14, 15]


def test_t64_reproduces_table1_medusa_row():
    rows = [list(map(int, l.split())) for l in open(os.path.join(HERE, "golden", "table1_medusa_row.txt"))
            if l.strip() and not l.startswith("#")]
    t = synth.t64()
    _check_tree(t, 4, (10,) * 4)
    assert _levels(t) == [1, 10, 23, 23, 7]
    for heads, leaves, nodes in rows:
        keep = t.depth <= heads
        sub_parent = t.parent[keep]
        has_kid = np.zeros(int(keep.sum()), bool)
        has_kid[sub_parent[1:]] = True
        assert (int(keep.sum()), int((~has_kid).sum())) == (nodes, leaves), heads


@pytest.mark.parametrize("n", [1, 2, 8, 16, 32, 64, 128])
def test_random_trees_valid(n):
    rng = np.random.default_rng(n)
    for _ in range(5):
        t = synth.random_tree(rng, n)
        assert t.n == n
        _check_tree(t, 4, (10,) * 4)


def test_chain_and_star():
    c = synth.chain_tree(5)
    assert c.parent.tolist() == [-1, 0, 1, 2, 3] and c.depth.tolist() == [0, 1, 2, 3, 4]
    s = synth.star_tree(5)
    assert s.parent.tolist() == [-1, 0, 0, 0, 0] and s.rank.tolist() == [0, 0, 1, 2, 3]


@pytest.mark.parametrize("cfg", [configs.TINY_FP32, configs.LLAMA2_13B])
def test_pool_layout(cfg):
    wl = synth.make(cfg, with_heads=False)
    canary = synth.CANARY_FP32 if cfg.dtype == "fp32" else synth.CANARY_BF16
    free = synth.FREE_FP32 if cfg.dtype == "fp32" else synth.FREE_BF16
    raw = wl.pool_k.view(np.uint32 if cfg.dtype == "fp32" else np.uint16)
    sizes = np.diff(wl.node_off)
    assert raw[:, 0, :].min() == canary == raw[:, 0, :].max()
    for b in range(cfg.B):
        s, L, N, c = int(wl.seq_base[b]), int(wl.lens[b]), int(sizes[b]), int(wl.seq_cap[b])
        assert L + N <= c
        assert np.all(raw[:, s - 1, :] == canary) and np.all(raw[:, s + c, :] == canary)
        assert np.all(raw[:, s + L + N:s + c, :] == free)
        assert not np.any(raw[:, s:s + L + N, :] == canary)
    assert wl.cap_total == int(wl.seq_base[-1] + wl.seq_cap[-1] + 1)


def test_budget_policies():
    wl = synth.make(configs.LLAMA2_70B, with_heads=False)
    live = wl.lens.astype(np.int64) + np.diff(wl.node_off)
    assert np.array_equal(wl.seq_cap, live + live // 10)
    assert np.all((wl.lens >= 512) & (wl.lens <= 4096))
    wl = synth.make(configs.LLAMA2_7B, with_heads=False)
    assert np.array_equal(wl.seq_cap, wl.lens + 64)


def test_stress_shapes():
    wl = synth.make(configs.STRESS, with_heads=False)
    sizes = np.diff(wl.node_off)
    assert set(sizes.tolist()) <= {8, 16, 32, 64, 128}
    assert np.all((wl.lens >= 256) & (wl.lens <= 16384))
    assert np.all((wl.p_accept >= 0.3) & (wl.p_accept <= 0.8))
    for t in wl.trees:
        _check_tree(t, 4, (10,) * 4)


def test_planted_walk_is_a_root_path():
    wl = synth.make(configs.LLAMA2_13B, with_heads=False)
    for b, (plan, path) in enumerate(zip(wl.plan, wl.plan_path)):
        t = wl.trees[b]
        assert path[0] == 0
        for u, c in zip(path[:-1], path[1:]):
            assert t.parent[c] == u
        his = [(u, c) for u, c, v in plan if v > 0]
        assert [c for _, c in his] == path[1:]
        los = [(u, c) for u, c, v in plan if v < 0]
        if los:
            assert {c for _, c in los} == set(synth.children(t, path[-1]))
        else:
            assert not synth.children(t, path[-1])


def test_model_parameter_counts():
    # Llama-2 decoder: q/o projections hidden^2, k/v hidden x (n_kv * d), a
    # gated MLP of three hidden x ffn matrices, two norms per layer, untied
    # embedding and output matrices and a final norm.
    ffn = {"llama2_7b_b1": 11008, "llama2_13b_b4": 13824, "llama2_70b_b10": 28672, "stress_b32": 28672}
    for name, f in ffn.items():
        c = configs.get(name)
        h, kv = c.hidden, c.n_kv * c.head_dim
        layer = 2 * h * h + 2 * h * kv + 3 * h * f + 2 * h
        assert c.params == c.layers * layer + 2 * c.vocab * h + h, name
