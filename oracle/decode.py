"""Multi-step decoding on the CPU oracle.  TEST INFRASTRUCTURE.

Chains verify steps the way a serving loop does (SpecMemo Sec. 3.1: the KV
cache is a preallocated scratch space, sized to a budget, updated after every
verification; Sec. 3.2 / Alg. 1: the tree is pruned right to left to what the
budget holds).  Per step, for the sequences whose slab still has room:

  1. tree size N_b = min(default nodes, free slab rows); the tree is the
     default tree's first N_b nodes; a full slab ends its sequence;
  2. the tree's K/V rows (the base model's, drawn by the input generator) are
     written at slab rows L_b ..;
  3. residual-block heads (when given), projection, top-k, tree tokens, with
     the previous step's next token as the root;
  4. the planted base-model logits, tree attention, greedy or typical
     acceptance (App. A.1), and the next token, the acceptance's or sampled
     (Gumbel-max with Philox);
  5. compaction; L_b grows by the accepted tokens, the next token becomes the
     next root.

Only the tests and the benchmark's CPU leg may import this module; it never
imports the HIP library or its binding.
"""

from __future__ import annotations

import numpy as np

import oracle
from oracle import budget
from paper_2506_01986_amd import synth


def _concat(trees):
    node_off = np.concatenate([[0], np.cumsum([t.n for t in trees])]).astype(np.int32)
    return (node_off, np.concatenate([t.parent for t in trees]).astype(np.int32),
            np.concatenate([t.depth for t in trees]).astype(np.int32),
            np.concatenate([t.rank for t in trees]).astype(np.int32))


def run(setup: synth.DecodeSetup, steps: int, attn_rows=None):
    """Run up to `steps` steps.  Returns (per-step records, final K, final V,
    final lengths).  attn_rows(step, sumN, n_q) may select the (node, head)
    pairs whose attention output is computed (all when it returns None)."""
    cfg = setup.cfg
    K, V = setup.pool_k.copy(), setup.pool_v.copy()
    lens = setup.lens.astype(np.int32).copy()
    root = setup.root_tok.copy()
    dp, dd, dr = (list(map(int, a)) for a in (setup.default.parent, setup.default.depth, setup.default.rank))
    stride = cfg.n_heads + 1
    records = []
    for t in range(steps):
        sizes = budget.plan_tree_sizes(list(lens), list(setup.seq_cap), len(dp))
        seqs = [b for b in range(cfg.B) if sizes[b] > 0]
        if not seqs:
            break
        trees = []
        for b in seqs:
            p, d, r = budget.prune_to(dp, dd, dr, sizes[b])
            trees.append(synth.Tree(np.array(p, np.int32), np.array(d, np.int32), np.array(r, np.int32)))
        inp = synth.decode_step_inputs(setup, t, seqs, trees)
        node_off, parent, depth, rank = _concat(trees)
        base, L = setup.seq_base[seqs], lens[seqs]
        for i, b in enumerate(seqs):
            o, n, s0 = int(node_off[i]), trees[i].n, int(base[i]) + int(L[i])
            K[:, s0:s0 + n] = inp.tree_k[:, o:o + n]
            V[:, s0:s0 + n] = inp.tree_v[:, o:o + n]
        if setup.w1 is not None:
            hh = oracle.to_storage(oracle.resblock(inp.hidden, setup.w1, setup.b1), cfg.dtype)
            z = np.concatenate([oracle.head_logits(hh[i], setup.head_w[i:i + 1]) for i in range(cfg.n_heads)],
                               axis=1)
        else:
            z = oracle.head_logits(inp.hidden, setup.head_w)
        ids, _ = oracle.heads_topk(z, cfg.topk, cfg.kmax)
        tok = oracle.tree_tokens(node_off, depth, rank, root[seqs], ids)
        lg = synth.plant_logits(inp.base_logits, node_off, inp.plans, tok, cfg.dtype)
        sel = attn_rows(t, int(node_off[-1]), cfg.n_q) if attn_rows else None
        out = oracle.tree_attn(inp.q, K, V, node_off, parent, L, base, cfg.n_kv, sel=sel)
        if setup.typical is not None:
            T, eps, delta = setup.typical
            acc, path, nxt = oracle.accept_typical(lg, tok, node_off, parent, depth, stride, T, eps, delta)
        else:
            acc, path, nxt = oracle.accept_greedy(lg, tok, node_off, parent, depth, stride)
        best = second = None
        if setup.temperature is not None:
            nxt, best, second = oracle.sample_next(lg, node_off, acc, path, setup.temperature,
                                                   setup.sample_seed, t)
        new_len = oracle.kv_compact(K, V, base, L, acc, path)
        lens[seqs] = new_len
        root[seqs] = nxt
        records.append(dict(step=t, seqs=seqs, sizes=[sizes[b] for b in seqs], z=z, ids=ids, tok=tok, sel=sel,
                            attn=out, acc=acc, path=path, next_tok=nxt, best_key=best, second_key=second,
                            lens=lens.copy()))
    return records, K, V, lens
