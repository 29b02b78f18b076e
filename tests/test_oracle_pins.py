"""Pins of the CPU oracle to facts that do not come from the oracle itself.

Each stage is checked against a closed form, a library routine applied to a
special case, an invariant, or brute-force enumeration on tiny inputs, so that
a dropped term, a wrong sign or index, or a transposed operand fails a test.
"""

import itertools
import os

import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch

import oracle
from paper_2506_01986_amd import configs, synth


def small_cfg(dtype="fp32", B=2, n_q=4, n_kv=2, d=16, vocab=64, hidden=32, n_heads=4,
              topk=(4, 3, 2, 2), seed=123):
    return configs.Config(name="pin", dtype=dtype, B=B, n_q=n_q, n_kv=n_kv, head_dim=d,
                          hidden=hidden, vocab=vocab, n_heads=n_heads, topk=topk, tree="T16",
                          kv_len=(8, 8), seed=seed, w_std=1.0)


def f64(x, dt):
    return synth.storage_to_f64(x, dt)


# ----------------------------------------------------------------------------
# head logits and top-k
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_head_logits_equal_float64_matmul(dtype):
    cfg = small_cfg(dtype=dtype, B=3, hidden=48, vocab=37, n_heads=3, topk=(4, 2, 2))
    wl = synth.make(cfg, trees=[synth.t16()] * 3, lens=[5, 6, 7])
    z = oracle.head_logits(wl.hidden, wl.head_w)
    ref = np.matmul(f64(wl.hidden, dtype)[:, None, None, :],
                    np.swapaxes(f64(wl.head_w, dtype), 1, 2)[None]).squeeze(2)
    assert z.shape == (3, 3, 37)
    assert np.allclose(z, ref, rtol=1e-12, atol=1e-12)
    zs = oracle.head_logits(wl.hidden, wl.head_w, bsel=[2, 0])
    assert np.array_equal(zs, z[[2, 0]])


def test_topk_equals_stable_sort_with_ties():
    rng = np.random.default_rng(0)
    z = rng.integers(0, 6, size=(50, 40)).astype(np.float64)   # many equal values
    z[:5] = rng.standard_normal((5, 40))
    ids, vals = oracle.topk(z, 7)
    ref = np.argsort(-z, axis=1, kind="stable")[:, :7]
    assert np.array_equal(ids, ref)
    assert np.array_equal(vals, np.take_along_axis(z, ref, 1))


def test_topk_full_width():
    z = np.array([[3.0, 1.0, 3.0, 2.0]])
    ids, _ = oracle.topk(z, 4)
    assert ids.tolist() == [[0, 2, 3, 1]]


@pytest.mark.parametrize("tree,topk", [("T16", (4, 2, 2)), ("T64", (10, 10, 10, 10))])
def test_tree_tokens_level_i_holds_head_i(tree, topk):
    t = synth.t16() if tree == "T16" else synth.t64()
    cfg = small_cfg(B=2, vocab=90, n_heads=len(topk), topk=topk)
    wl = synth.make(cfg, trees=[t, t], lens=[4, 4])
    z = oracle.head_logits(wl.hidden, wl.head_w)
    ids, _ = oracle.heads_topk(z, topk, max(topk))
    tok = oracle.tree_tokens(wl.node_off, wl.depth, wl.rank, wl.root_tok, ids)
    for b in range(2):
        o = wl.node_off[b]
        assert tok[o] == wl.root_tok[b]
        level1 = [n for n in range(t.n) if t.depth[n] == 1]
        # the root's children, in BFS order, carry head 0's top-k in decreasing logit order
        assert tok[o + np.array(level1)].tolist() == \
            np.argsort(-z[b, 0], kind="stable")[:len(level1)].tolist()
        for n in range(1, t.n):
            if t.rank[n] == 0:     # rank 0 at depth i is head i-1's argmax
                assert tok[o + n] == int(np.argmax(z[b, t.depth[n] - 1]))


# ----------------------------------------------------------------------------
# tree attention
# ----------------------------------------------------------------------------

def ancestor_closure(parent):
    """anc_or_self[n, j] via powers of the child->parent adjacency matrix."""
    n = len(parent)
    P = np.zeros((n, n))
    for c in range(1, n):
        P[c, parent[c]] = 1.0
    R, M = np.eye(n), np.eye(n)
    for _ in range(n):
        M = M @ P
        R += M
    return R > 0


def sdpa(Q, K, V, mask):
    out = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q)[None, None], torch.from_numpy(K)[None, None],
        torch.from_numpy(V)[None, None], attn_mask=torch.from_numpy(mask))
    return out[0, 0].numpy()


def sdpa_tree(wl, b, h, tree_mask):
    cfg = wl.cfg
    kv = h // (cfg.n_q // cfg.n_kv)
    o, N, L, s0 = int(wl.node_off[b]), wl.trees[b].n, int(wl.lens[b]), int(wl.seq_base[b])
    dt = cfg.dtype
    Q = f64(wl.q[o:o + N, h, :], dt)
    K = f64(wl.pool_k[kv, s0:s0 + L + N, :], dt)
    V = f64(wl.pool_v[kv, s0:s0 + L + N, :], dt)
    mask = np.concatenate([np.ones((N, L), bool), tree_mask], axis=1)
    return sdpa(Q, K, V, mask)


def run_attn(wl, **kw):
    return oracle.tree_attn(wl.q, wl.pool_k, wl.pool_v, wl.node_off, wl.parent, wl.lens,
                            wl.seq_base, wl.cfg.n_kv, **kw)


@pytest.mark.parametrize("dtype,n_q,n_kv", [("fp32", 4, 4), ("bf16", 8, 2)])
def test_chain_tree_is_causal_attention(dtype, n_q, n_kv):
    N = 5
    cfg = small_cfg(dtype=dtype, B=2, n_q=n_q, n_kv=n_kv)
    wl = synth.make(cfg, trees=[synth.chain_tree(N)] * 2, lens=[9, 0])
    out = run_attn(wl)
    causal = np.tril(np.ones((N, N), bool))
    for b in range(2):
        for h in range(n_q):
            ref = sdpa_tree(wl, b, h, causal)
            o = wl.node_off[b]
            assert np.allclose(out[o:o + N, h], ref, rtol=1e-12, atol=1e-13)


def test_single_node_is_decode_attention():
    cfg = small_cfg(B=3, n_q=4, n_kv=1)
    wl = synth.make(cfg, trees=[synth.tree_from_rank_paths([()])] * 3, lens=[1, 13, 40])
    out = run_attn(wl)
    for b in range(3):
        L, s0 = int(wl.lens[b]), int(wl.seq_base[b])
        for h in range(4):
            Q = wl.q[b:b + 1, h].astype(np.float64)
            K = wl.pool_k[0, s0:s0 + L + 1].astype(np.float64)
            V = wl.pool_v[0, s0:s0 + L + 1].astype(np.float64)
            ref = torch.nn.functional.scaled_dot_product_attention(
                *(torch.from_numpy(x)[None, None] for x in (Q, K, V)))[0, 0].numpy()
            assert np.allclose(out[b, h], ref[0], rtol=1e-12, atol=1e-13)


def test_star_tree_node_sees_root_and_itself():
    N = 7
    cfg = small_cfg(B=1, n_q=2, n_kv=2, topk=(8, 2, 2, 2))
    wl = synth.make(cfg, trees=[synth.star_tree(N)], lens=[6])
    out = run_attn(wl)
    mask = np.eye(N, dtype=bool)
    mask[:, 0] = True
    for h in range(2):
        assert np.allclose(out[:, h], sdpa_tree(wl, 0, h, mask), rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("n", [3, 16, 64, 128])
def test_random_trees_match_masked_sdpa(n):
    rng = np.random.default_rng(n)
    trees = [synth.random_tree(rng, n), synth.random_tree(rng, max(1, n // 2))]
    cfg = small_cfg(dtype="bf16", B=2, n_q=4, n_kv=2, topk=(10,) * 4)
    wl = synth.make(cfg, trees=trees, lens=[3, 17])
    out = run_attn(wl)
    for b in range(2):
        m = ancestor_closure(wl.trees[b].parent)
        o, N = wl.node_off[b], wl.trees[b].n
        for h in range(4):
            assert np.allclose(out[o:o + N, h], sdpa_tree(wl, b, h, m), rtol=1e-12, atol=1e-13)


def test_gqa_equals_mha_with_repeated_kv():
    cfg = small_cfg(dtype="bf16", B=2, n_q=8, n_kv=2)
    wl = synth.make(cfg, trees=[synth.t16(), synth.random_tree(np.random.default_rng(1), 9)],
                    lens=[11, 4])
    out = run_attn(wl)
    K = np.ascontiguousarray(np.repeat(wl.pool_k, 4, axis=0))   # kv head j -> q heads 4j..4j+3
    V = np.ascontiguousarray(np.repeat(wl.pool_v, 4, axis=0))
    out_mha = oracle.tree_attn(wl.q, K, V, wl.node_off, wl.parent, wl.lens, wl.seq_base, 8)
    assert np.array_equal(out, out_mha)


def test_committed_row_permutation_invariance():
    cfg = small_cfg(B=1)
    wl = synth.make(cfg, trees=[synth.t16()], lens=[12])
    out = run_attn(wl)
    s0 = int(wl.seq_base[0])
    perm = np.random.default_rng(3).permutation(12)
    for pool in (wl.pool_k, wl.pool_v):
        pool[:, s0:s0 + 12] = pool[:, s0 + perm]
    assert np.allclose(run_attn(wl), out, rtol=1e-12, atol=1e-13)


def test_uniform_values_give_uniform_output():
    cfg = small_cfg(B=2)
    wl = synth.make(cfg, trees=[synth.t16(), synth.chain_tree(4)], lens=[5, 0])
    for b in range(2):
        s0, L, N = int(wl.seq_base[b]), int(wl.lens[b]), wl.trees[b].n
        wl.pool_v[:, s0:s0 + L + N] = 1.0
    assert np.allclose(run_attn(wl), 1.0, rtol=0, atol=1e-14)


def test_common_key_shift_invariance():
    cfg = small_cfg(B=1)
    wl = synth.make(cfg, trees=[synth.t16()], lens=[10])
    out = run_attn(wl)
    s0 = int(wl.seq_base[0])
    u = np.random.default_rng(4).standard_normal((cfg.n_kv, 1, cfg.head_dim)).astype(np.float32)
    wl.pool_k[:, s0:s0 + 10 + 16] += u      # every key of the slab moves by the same vector
    assert np.allclose(run_attn(wl), out, rtol=1e-5, atol=1e-6)


def test_explicit_scale_and_selection():
    cfg = small_cfg(B=2)
    wl = synth.make(cfg, trees=[synth.t16(), synth.chain_tree(3)], lens=[5, 2])
    full = run_attn(wl, scale=0.3)
    sel = np.array([[17, 3], [0, 0], [5, 1]])
    part = run_attn(wl, scale=0.3, sel=sel)
    for i, (n, h) in enumerate(sel):
        assert np.array_equal(part[i], full[n, h])
    # scale 0 makes every visible key equally likely: the output is their mean
    z = run_attn(wl, scale=0.0)
    s0, L = int(wl.seq_base[1]), int(wl.lens[1])
    o = wl.node_off[1]
    for n in range(3):                       # chain: node n sees tree rows 0..n
        rows = list(range(L)) + [L + j for j in range(n + 1)]
        ref = wl.pool_v[0, s0 + np.array(rows)].astype(np.float64).mean(0)
        assert np.allclose(z[o + n, 0], ref, rtol=1e-12, atol=1e-13)


# ----------------------------------------------------------------------------
# acceptance
# ----------------------------------------------------------------------------

def brute_accept(logits, tok, parent, mode, T=1.0, eps=0.0, delta=0.0):
    """Enumerate every root-to-leaf path; take its longest accepted prefix;
    keep the best prefix by (length, sum log pi, -last node id)."""
    N = len(parent)
    kids = {u: [c for c in range(N) if parent[c] == u] for u in range(N)}
    leaves = [u for u in range(N) if not kids[u]]
    logp = logits / T - scipy.special.logsumexp(logits / T, axis=1, keepdims=True)
    ent = scipy.stats.entropy(scipy.special.softmax(logits / T, axis=1), axis=1)
    best = None
    for leaf in leaves:
        p = [leaf]
        while p[-1] != 0:
            p.append(parent[p[-1]])
        p = p[::-1]
        j, score = 0, 0.0
        for u, c in zip(p[:-1], p[1:]):
            if mode == "greedy":
                ok = int(np.argmax(logits[u])) == tok[c]
            else:
                ok = np.exp(logp[u, tok[c]]) > min(eps, delta * np.exp(-ent[u]))
            if not ok:
                break
            j += 1
            score += logp[u, tok[c]]
        key = (j, score if mode == "typical" else 0.0, -p[j])
        if best is None or key > best[0]:
            best = (key, p[:j + 1])
    path = best[1]
    return len(path) - 1, path, int(np.argmax(logits[path[-1]]))


def tiny_case(rng, vocab, int_logits):
    n = int(rng.integers(1, 13))
    t = synth.random_tree(rng, n, max_depth=4, max_kids=min(4, vocab))
    tok = np.zeros(n, np.int32)
    tok[0] = rng.integers(vocab)
    for u in range(n):
        kids = synth.children(t, u)
        tok[kids] = rng.choice(vocab, size=len(kids), replace=False)
    if int_logits:
        lg = rng.integers(0, 3, size=(n, vocab)).astype(np.float32)
    else:
        lg = (2.0 * rng.standard_normal((n, vocab))).astype(np.float32)
    return t, tok, lg


@pytest.mark.parametrize("int_logits", [True, False])
def test_greedy_acceptance_equals_brute_force(int_logits):
    rng = np.random.default_rng(11 + int_logits)
    for _ in range(300):
        vocab = int(rng.integers(2, 7))
        t, tok, lg = tiny_case(rng, vocab, int_logits)
        acc, path, nxt = oracle.accept_greedy(lg, tok, [0, t.n], t.parent, t.depth, 6)
        ra, rp, rn = brute_accept(lg.astype(np.float64), tok, t.parent, "greedy")
        assert acc[0] == ra and nxt[0] == rn
        assert path[0, :ra + 1].tolist() == rp and np.all(path[0, ra + 1:] == -1)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_softmax_stats_equal_library_logsumexp_and_entropy(dtype):
    rng = np.random.default_rng(41)
    raw = (rng.standard_normal((6, 32000)) * np.array([[1.0], [3.0], [0.1], [1.0], [8.0], [1.0]])).astype(np.float32)
    raw[3, 17] = 200.0                                    # one dominant token: entropy near 0
    raw[5] = 2.5                                          # uniform row: lse = x + log w, H = log w
    z = synth._store(raw.reshape(-1), dtype).reshape(raw.shape)
    x64 = f64(z, dtype)
    for T in (0.7, 1.0, 1.5):
        lse, ent = oracle.softmax_stats(z, T)
        assert np.allclose(lse, scipy.special.logsumexp(x64 / T, axis=1), rtol=1e-13, atol=1e-12)
        assert np.allclose(ent, scipy.stats.entropy(scipy.special.softmax(x64 / T, axis=1), axis=1),
                           rtol=1e-11, atol=1e-12)
        assert abs(ent[5] - np.log(32000)) < 1e-12 and abs(lse[5] - (2.5 / T + np.log(32000))) < 1e-12
        assert ent[3] < 1e-10


def test_typical_acceptance_equals_brute_force():
    rng = np.random.default_rng(5)
    for i in range(300):
        vocab = int(rng.integers(3, 9))
        t, tok, lg = tiny_case(rng, vocab, int_logits=False)
        T, eps, delta = 0.7, float(rng.uniform(0.05, 0.4)), float(rng.uniform(0.1, 0.9))
        acc, path, nxt = oracle.accept_typical(lg, tok, [0, t.n], t.parent, t.depth, 6, T, eps, delta)
        ra, rp, rn = brute_accept(lg.astype(np.float64), tok, t.parent, "typical", T, eps, delta)
        assert (acc[0], path[0, :ra + 1].tolist(), nxt[0]) == (ra, rp, rn), i


def test_typical_tie_breaks():
    # root -> children 1, 2 (depth 1, leaves).  Both edges pass.
    parent = np.array([-1, 0, 0], np.int32)
    depth = np.array([0, 1, 1], np.int32)
    tok = np.array([0, 3, 1], np.int32)
    lg = np.zeros((3, 6), np.float32)
    lg[0, [1, 3]] = 4.0                  # equal probabilities: the lower node id (1) wins
    acc, path, _ = oracle.accept_typical(lg, tok, [0, 3], parent, depth, 3, 1.0, 0.09, 0.3)
    assert acc[0] == 1 and path[0].tolist() == [0, 1, -1]
    lg[0, 1] = 4.5                       # node 2's token is now more likely: node 2 wins
    acc, path, _ = oracle.accept_typical(lg, tok, [0, 3], parent, depth, 3, 1.0, 0.09, 0.3)
    assert acc[0] == 1 and path[0].tolist() == [0, 2, -1]


def node_tokens_distinct(wl, rng):
    tok = np.zeros(wl.total_nodes, np.int32)
    for b, t in enumerate(wl.trees):
        o = wl.node_off[b]
        tok[o] = wl.root_tok[b]
        for u in range(t.n):
            kids = synth.children(t, u)
            tok[o + np.array(kids, int)] = rng.choice(wl.cfg.vocab, size=len(kids), replace=False)
    return tok


@pytest.mark.parametrize("mode", ["greedy", "typical"])
def test_planted_walk_is_accepted(mode):
    for cfg in (configs.TINY_FP32, configs.LLAMA2_13B):
        wl = synth.make(cfg, with_heads=cfg is configs.TINY_FP32)
        if wl.head_w is not None:
            z = oracle.head_logits(wl.hidden, wl.head_w)
            ids, _ = oracle.heads_topk(z, cfg.topk, cfg.kmax)
            tok = oracle.tree_tokens(wl.node_off, wl.depth, wl.rank, wl.root_tok, ids)
        else:
            tok = node_tokens_distinct(wl, np.random.default_rng(0))
        lg = synth.planted_logits(wl, tok)
        stride = cfg.n_heads + 1
        if mode == "greedy":
            acc, path, nxt = oracle.accept_greedy(lg, tok, wl.node_off, wl.parent, wl.depth, stride)
        else:
            acc, path, nxt = oracle.accept_typical(lg, tok, wl.node_off, wl.parent, wl.depth,
                                                   stride, 0.7, 0.09, 0.3)
        full = synth.storage_to_f64(lg, cfg.dtype)
        for b in range(cfg.B):
            want = wl.plan_path[b]
            assert acc[b] == len(want) - 1
            assert path[b, :len(want)].tolist() == want
            assert nxt[b] == int(np.argmax(full[wl.node_off[b] + want[-1]]))


# ----------------------------------------------------------------------------
# compaction
# ----------------------------------------------------------------------------

def _compaction_case(dtype):
    cfg = small_cfg(dtype=dtype, B=3, n_kv=2, n_q=4)
    wl = synth.make(cfg, trees=[synth.t16(), synth.chain_tree(5), synth.t16()], lens=[6, 0, 9])
    paths = np.full((3, 5), -1, np.int32)
    paths[0, :4] = [0, 2, 7, 14]          # overlapping: dest 2 is also the source of dest 1
    paths[1, :5] = [0, 1, 2, 3, 4]        # identity
    paths[2, :1] = [0]                    # root only
    acc = np.array([3, 4, 0], np.int32)
    return wl, acc, paths


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_compaction_moves_accepted_rows_only(dtype):
    wl, acc, paths = _compaction_case(dtype)
    K0, V0 = wl.pool_k.copy(), wl.pool_v.copy()
    K, V = wl.pool_k.copy(), wl.pool_v.copy()
    new_len = oracle.kv_compact(K, V, wl.seq_base, wl.lens, acc, paths)
    assert new_len.tolist() == (wl.lens + acc + 1).tolist()
    touched = np.zeros(wl.cap_total, bool)
    for b in range(3):
        s0, L = int(wl.seq_base[b]), int(wl.lens[b])
        for j in range(acc[b] + 1):
            for P, P0 in ((K, K0), (V, V0)):
                assert np.array_equal(P[:, s0 + L + j].view(np.uint8),
                                      P0[:, s0 + L + paths[b, j]].view(np.uint8))
            touched[s0 + L + j] = True
    for P, P0 in ((K, K0), (V, V0)):
        assert np.array_equal(P[:, ~touched].view(np.uint8), P0[:, ~touched].view(np.uint8))


# ----------------------------------------------------------------------------
# padded batching (Sec. 3.3): pad tokens in the cache, masked with -inf
# ----------------------------------------------------------------------------

def _padded_case(dtype, seed=5):
    rng = np.random.default_rng(seed)
    trees = [synth.random_tree(rng, 12), synth.t16(), synth.chain_tree(4)]
    cfg = small_cfg(dtype=dtype, B=3, n_q=4, n_kv=2, topk=(10,) * 4, seed=seed)
    wl = synth.make(cfg, trees=trees, lens=[40, 0, 23])
    valid = (rng.random(wl.cap_total) < 0.6).astype(np.uint8)
    for b in range(3):                    # tree rows are never consulted: make them pads too
        s0, L = int(wl.seq_base[b]), int(wl.lens[b])
        valid[s0 + L:s0 + L + wl.trees[b].n] = 0
    return wl, valid


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_padded_attention_equals_attention_without_pad_rows(dtype):
    # A key masked with -inf has weight exp(-inf) = 0: attention over a cache
    # with pad tokens equals attention over the same cache with them deleted.
    wl, valid = _padded_case(dtype)
    out = run_attn(wl, key_valid=valid)
    K, V = wl.pool_k.copy(), wl.pool_v.copy()
    lens = wl.lens.copy()
    for b in range(3):
        s0, L, N = int(wl.seq_base[b]), int(wl.lens[b]), wl.trees[b].n
        keep = [s0 + t for t in range(L) if valid[s0 + t]] + list(range(s0 + L, s0 + L + N))
        for P, P0 in ((K, wl.pool_k), (V, wl.pool_v)):
            P[:, s0:s0 + len(keep)] = P0[:, keep]
        lens[b] = len(keep) - N
    assert lens.tolist() != wl.lens.tolist()
    ref = oracle.tree_attn(wl.q, K, V, wl.node_off, wl.parent, lens, wl.seq_base, wl.cfg.n_kv)
    assert np.allclose(out, ref, rtol=1e-12, atol=1e-13)
    # all rows valid: the unpadded result, bit for bit
    full = run_attn(wl, key_valid=np.ones(wl.cap_total, np.uint8))
    assert np.array_equal(full, run_attn(wl))


def _golden_fig8():
    rows = [list(map(int, ln.split())) for ln in open(os.path.join(os.path.dirname(__file__), "golden",
                                                                   "fig8_padded_batch.txt"))
            if ln.strip() and not ln.startswith("#")]
    return np.array(rows)


def test_fig8_padding_of_accepted_tokens():
    from oracle import padded
    g = _golden_fig8()
    tau = g[:, 1]
    cfg = small_cfg(B=4, n_q=2, n_kv=2, topk=(10,) * 4)
    wl = synth.make(cfg, trees=[synth.chain_tree(5)] * 4, lens=[3, 0, 7, 1],
                    caps=[3 + 9, 9, 7 + 9, 1 + 9])
    acc = (tau - 1).astype(np.int32)
    paths = np.full((4, 5), -1, np.int32)
    for b in range(4):
        paths[b, :tau[b]] = np.arange(tau[b])
    valid = np.ones(wl.cap_total, np.uint8)
    K, V = wl.pool_k.copy(), wl.pool_v.copy()
    pos0 = np.array([3, 0, 7, 1], np.int32)
    new_len, new_pos = padded.pad_update(K, V, wl.seq_base, wl.lens, pos0, valid, acc, paths)
    uniform = int(g[0, 1] + g[0, 2])               # accepted + pads, the same for every sequence
    assert (g[:, 1] + g[:, 2]).tolist() == [uniform] * 4
    assert (new_len - wl.lens).tolist() == [uniform] * 4
    assert (new_pos - pos0).tolist() == tau.tolist()
    for b in range(4):
        s0, L = int(wl.seq_base[b]), int(wl.lens[b])
        assert valid[s0 + L:s0 + L + uniform].tolist() == [1] * tau[b] + [0] * g[b, 2]
    # the chain paths are identities: no K/V row moves
    assert np.array_equal(K.view(np.uint8), wl.pool_k.view(np.uint8))


def test_padded_steps_keep_the_tokens_of_compaction():
    # Three decode steps from one state, once compacted and once padded, with
    # the same accepted paths and the same fresh tree K/V each step: the
    # non-pad rows of each padded slab, in order, are the compacted slab's
    # committed rows, and the position equals the compacted length.
    from oracle import padded
    rng = np.random.default_rng(9)
    trees = [synth.t16(), synth.random_tree(rng, 20, max_depth=3), synth.chain_tree(4)]
    cfg = small_cfg(dtype="bf16", B=3, n_q=4, n_kv=2, topk=(10,) * 4)
    lens0 = np.array([5, 0, 11], np.int32)
    caps = lens0 + 80
    wl = synth.make(cfg, trees=trees, lens=lens0, caps=caps)
    Kc, Vc = wl.pool_k.copy(), wl.pool_v.copy()
    Kp, Vp = wl.pool_k.copy(), wl.pool_v.copy()
    valid = np.ones(wl.cap_total, np.uint8)
    Lc, Lp, pos = lens0.copy(), lens0.copy(), lens0.copy()
    for step in range(3):
        acc = np.zeros(3, np.int32)
        paths = np.full((3, 5), -1, np.int32)
        for b, t in enumerate(trees):
            walk = [0]
            while True:
                kids = synth.children(t, walk[-1])
                if not kids or rng.random() < 0.3:
                    break
                walk.append(kids[int(rng.integers(len(kids)))])
            acc[b] = len(walk) - 1
            paths[b, :len(walk)] = walk
            s0, N = int(wl.seq_base[b]), t.n
            fresh = rng.integers(0, 1 << 16, size=(2, cfg.n_kv, N, cfg.head_dim)).astype(np.uint16)
            Kc[:, s0 + Lc[b]:s0 + Lc[b] + N], Vc[:, s0 + Lc[b]:s0 + Lc[b] + N] = fresh[0], fresh[1]
            Kp[:, s0 + Lp[b]:s0 + Lp[b] + N], Vp[:, s0 + Lp[b]:s0 + Lp[b] + N] = fresh[0], fresh[1]
        Lc = oracle.kv_compact(Kc, Vc, wl.seq_base, Lc, acc, paths)
        Lp, pos = padded.pad_update(Kp, Vp, wl.seq_base, Lp, pos, valid, acc, paths)
    assert pos.tolist() == Lc.tolist() and np.all(Lp >= Lc)
    for b in range(3):
        s0 = int(wl.seq_base[b])
        real = [s0 + r for r in range(int(Lp[b])) if valid[s0 + r]]
        assert len(real) == Lc[b]
        for Pp, Pc in ((Kp, Kc), (Vp, Vc)):
            assert np.array_equal(Pp[:, real].view(np.uint8), Pc[:, s0:s0 + Lc[b]].view(np.uint8))


# ----------------------------------------------------------------------------
# decode loop pieces: residual-block heads, Philox, sampled next token
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_resblock_equals_torch_linear_silu(dtype):
    rng = np.random.default_rng(31)
    B, hidden, n_heads = 3, 24, 2
    h = synth._store(rng.standard_normal(B * hidden).astype(np.float32), dtype).reshape(B, hidden)
    W1 = synth._store((0.3 * rng.standard_normal(n_heads * hidden * hidden)).astype(np.float32),
                      dtype).reshape(n_heads, hidden, hidden)
    b1 = synth._store(rng.standard_normal(n_heads * hidden).astype(np.float32), dtype).reshape(n_heads, hidden)
    out = oracle.resblock(h, W1, b1)
    H, W, bb = (torch.from_numpy(f64(x, dtype)) for x in (h, W1, b1))
    for i in range(n_heads):
        ref = H + torch.nn.functional.silu(torch.nn.functional.linear(H, W[i], bb[i]))
        assert np.allclose(out[i], ref.numpy(), rtol=1e-13, atol=1e-13)
    # zero weights and bias: the block is the identity
    z = np.zeros_like(W1), np.zeros_like(b1)
    assert np.array_equal(oracle.resblock(h, *z), np.broadcast_to(f64(h, dtype), out.shape))


def test_storage_rounding_equals_torch():
    rng = np.random.default_rng(32)
    x = np.concatenate([rng.standard_normal(10000) * 10.0 ** rng.integers(-8, 8, 10000),
                        [0.0, -0.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -9, 65504.0, 1e-30]])
    bf = oracle.to_storage(x, "bf16")
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bf, ref)
    assert np.array_equal(oracle.to_storage(x, "fp32"), x.astype(np.float32))


def _plus_one(ctr):
    c = [int(v) for v in ctr]
    for i in range(4):
        c[i] = (c[i] + 1) % (1 << 64)
        if c[i] != 0:
            break
    return c


@pytest.mark.parametrize("key,ctr", [((0, 0), (0, 0, 0, 0)), ((123456789, 987654321), (5, 6, 7, 8)),
                                     ((2 ** 64 - 1, 2 ** 63), (2 ** 64 - 1, 2 ** 64 - 1, 3, 4))])
def test_philox_equals_numpy_stream(key, ctr):
    # numpy's Philox (4 x 64 bits, 10 rounds) advances its counter before each
    # block of four outputs
    bg = np.random.Philox(key=np.array(key, np.uint64), counter=np.array(ctr, np.uint64))
    raw = bg.random_raw(12).reshape(3, 4)
    c = list(ctr)
    for blk in range(3):
        c = _plus_one(c)
        got = oracle.philox4x64_10(np.array([c], np.uint64), np.array([key], np.uint64))[0]
        assert np.array_equal(got, raw[blk]), blk


def _sample_rows(z, n, temperature, seed, offset):
    """n single-node sequences whose only row is z."""
    vocab = len(z)
    logits = np.tile(np.asarray(z, np.float32), (n, 1))
    node_off = np.arange(n + 1, dtype=np.int32)
    acc = np.zeros(n, np.int32)
    path = np.zeros((n, 1), np.int32)
    return oracle.sample_next(logits, node_off, acc, path, temperature, seed, offset)


@pytest.mark.parametrize("temperature", [0.5, 1.0, 2.5])
def test_sampled_token_follows_softmax(temperature):
    z = np.array([0.3, -1.2, 2.0, 0.0, 1.1, -0.4], np.float32)
    n = 40000
    tok, _, _ = _sample_rows(z, n, temperature, seed=77, offset=3)
    counts = np.bincount(tok, minlength=len(z))
    p = scipy.special.softmax(z.astype(np.float64) / temperature)
    chi = scipy.stats.chisquare(counts, n * p)
    assert chi.pvalue > 1e-3, (counts, n * p)
    # another seed or offset draws other tokens
    assert not np.array_equal(tok, _sample_rows(z, n, temperature, seed=78, offset=3)[0])
    assert not np.array_equal(tok, _sample_rows(z, n, temperature, seed=77, offset=4)[0])


def test_sampling_at_low_temperature_is_argmax():
    rng = np.random.default_rng(33)
    z = rng.standard_normal(257).astype(np.float32)
    tok, _, _ = _sample_rows(z, 50, 1e-4, seed=1, offset=0)
    assert np.all(tok == int(np.argmax(z)))


def test_sampling_reads_the_last_accepted_row():
    # three single-path trees of 4 nodes; each node's row puts a dominant logit
    # on a token of its own, so the draw names the row that was read
    B, n, vocab = 3, 4, 50
    logits = np.zeros((B * n, vocab), np.float32)
    for r in range(B * n):
        logits[r, r] = 60.0
    node_off = np.arange(0, B * n + 1, n, dtype=np.int32)
    acc = np.array([0, 3, 2], np.int32)
    path = np.tile(np.arange(n, dtype=np.int32), (B, 1))
    tok, _, _ = oracle.sample_next(logits, node_off, acc, path, 1.0, 5, 0)
    assert tok.tolist() == [0 * n + 0, 1 * n + 3, 2 * n + 2]


def test_gumbel_words_give_finite_standard_gumbel_values():
    # Every 64-bit word maps to a finite value: the extreme words (all zeros,
    # all ones) included, where a 24-bit uniform rounded in fp32 would reach
    # u = 1 and G = +inf.  Only the top 23 bits count, and G grows with them.
    extremes = np.array([0, 2 ** 64 - 1, 2 ** 41 - 1, 2 ** 63, (2 ** 23 - 1) << 41], np.uint64)
    g = oracle.gumbel(extremes)
    assert np.all(np.isfinite(g))
    assert g[0] == g[2] and g[1] == g[4]
    assert g[0] < g[3] < g[1]
    # The 2^23 equally likely top-bit patterns form a midpoint grid over (0, 1):
    # the mean and variance of -log(-log u) over it are the standard Gumbel
    # law's, Euler's constant and pi^2 / 6 (closed forms), up to the grid error.
    k = np.arange(2 ** 23, dtype=np.uint64) << np.uint64(41)
    gg = oracle.gumbel(k)
    assert np.all(np.diff(gg) > 0)
    assert abs(gg.mean() - np.euler_gamma) < 1e-5
    assert abs(gg.var() - np.pi ** 2 / 6) < 1e-3
