"""Pins of the oracle's multi-step decode loop (oracle.decode): the budget
rule for tree sizes, the cache holding exactly the accepted tokens' K/V rows
in order, the planted walks accepted, and the token chain between steps."""

import numpy as np
import pytest

from oracle import decode
from paper_2506_01986_amd import configs, synth


def _cfg(dtype="bf16", **kw):
    base = dict(name="dec", dtype=dtype, B=3, n_q=4, n_kv=2, head_dim=32, hidden=48, vocab=300, n_heads=4,
                topk=(10, 10, 10, 10), tree="T64", kv_len=(5, 30), kv_len_dist="uniform", seed=5,
                w_std=0.05 if dtype == "bf16" else 1.0, p_accept=0.7)
    base.update(kw)
    return configs.Config(**base)


@pytest.mark.parametrize("resblock,temperature,typical", [(False, None, None), (True, None, None), (True, 0.8, None),
                                                          (True, None, (0.7, 0.09, 0.3))])
def test_decode_loop_bookkeeping(resblock, temperature, typical):
    cfg = _cfg()
    default = synth.t64()
    room = [200, 70, 9]                     # the third slab fills up within a few steps, the second shrinks its trees
    st = synth.decode_setup(cfg, 5, default, room, resblock=resblock, temperature=temperature, typical=typical)
    recs, K, V, lens = decode.run(st, 12)
    L = st.lens.astype(np.int64).copy()
    expect_rows = {b: [(st.pool_k[:, int(st.seq_base[b]) + r], st.pool_v[:, int(st.seq_base[b]) + r])
                       for r in range(int(L[b]))] for b in range(cfg.B)}
    root = st.root_tok.copy()
    shrank = False
    for rec in recs:
        t, seqs = rec["step"], rec["seqs"]
        # tree size: the default tree cut to the slab's free rows
        for b, n in zip(seqs, rec["sizes"]):
            assert n == min(default.n, int(st.seq_cap[b]) - int(L[b])) and n > 0
            shrank |= n < default.n
        for b in range(cfg.B):
            if b not in seqs:
                assert int(st.seq_cap[b]) - int(L[b]) <= 0
        # the step's trees and inputs, regenerated
        trees = [synth.tree_prefix(default, n) for n in rec["sizes"]]
        inp = synth.decode_step_inputs(st, t, seqs, trees)
        off = np.concatenate([[0], np.cumsum([tr.n for tr in trees])])
        tok = rec["tok"]
        for i, b in enumerate(seqs):
            o = int(off[i])
            assert tok[o] == root[b]                                   # the previous step's next token
            acc = int(rec["acc"][i])
            path = rec["path"][i, :acc + 1]
            # greedy or typical acceptance of planted logits follows the planted walk
            planted = [0] + [c for (u, c, v) in inp.plans[i] if v > 0]
            assert path.tolist() == planted
            # the accepted tree rows, in path order, join the committed rows
            for j in path:
                expect_rows[b].append((inp.tree_k[:, o + int(j)], inp.tree_v[:, o + int(j)]))
            L[b] += acc + 1
            root[b] = rec["next_tok"][i]
            if temperature is None:
                assert rec["next_tok"][i] >= 0
        assert rec["lens"].tolist() == L.tolist()
    assert shrank, "no tree was pruned by the budget"
    assert L[2] == st.seq_cap[2] and 2 not in recs[-1]["seqs"], "the small slab did not fill up"
    assert len(recs) == 12
    for b in range(cfg.B):
        s0 = int(st.seq_base[b])
        assert len(expect_rows[b]) == lens[b] <= st.seq_cap[b]
        for r, (k, v) in enumerate(expect_rows[b]):
            assert np.array_equal(K[:, s0 + r].view(np.uint16), np.asarray(k).view(np.uint16)), (b, r)
            assert np.array_equal(V[:, s0 + r].view(np.uint16), np.asarray(v).view(np.uint16)), (b, r)


def test_sampled_tokens_differ_from_greedy_and_follow_the_seed():
    cfg = _cfg()
    st_g = synth.decode_setup(cfg, 6, synth.t64(), [400] * 3, resblock=False, temperature=None)
    st_s = synth.decode_setup(cfg, 6, synth.t64(), [400] * 3, resblock=False, temperature=5.0)
    rg, *_ = decode.run(st_g, 3)
    rs, *_ = decode.run(st_s, 3)
    # the first step's acceptance does not depend on the next-token rule
    assert np.array_equal(rg[0]["acc"], rs[0]["acc"])
    assert not np.array_equal(rg[0]["next_tok"], rs[0]["next_tok"])
    again, *_ = decode.run(st_s, 3)
    assert all(np.array_equal(a["next_tok"], b["next_tok"]) for a, b in zip(rs, again))


def test_typical_with_vanishing_thresholds_accepts_the_deepest_nodes():
    # with eps and delta near zero every edge passes typical acceptance, so each
    # step accepts a deepest node of its tree; greedy acceptance follows the
    # planted walks, which mostly stop earlier
    cfg = _cfg()
    common = dict(resblock=False, temperature=None)
    st_t = synth.decode_setup(cfg, 8, synth.t64(), [400] * 3, typical=(0.7, 1e-30, 1e-30), **common)
    st_g = synth.decode_setup(cfg, 8, synth.t64(), [400] * 3, **common)
    rt, *_ = decode.run(st_t, 3)
    rg, *_ = decode.run(st_g, 3)
    for rec in rt:
        for n, a in zip(rec["sizes"], rec["acc"]):
            assert a == int(synth.tree_prefix(st_t.default, n).depth.max())
    assert any(int(a) < 4 for rec in rg for a in rec["acc"])
