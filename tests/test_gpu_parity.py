"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Integers (top-k ids, node tokens, accepted lengths, paths, next tokens,
compaction results) must match bit-exactly; floats within |gpu - ref| <=
atol + rtol * |ref| with (1e-2, 2e-2) for bf16 and (1e-5, 1e-5) for fp32.

Top-k ids come from fp32 logits on the GPU and fp64 logits in the oracle.
Every logit must lie within tau = 1e-5 (1 + |z|) of the oracle's (an fp32
accumulation bound, tests/ties.py), and before the GPU runs, the hidden state
of any sequence whose k+1 largest fp64 logits of some head hold two within
2 tau is re-drawn (the re-draws are printed).  Every top-k id and tree token
is then compared with the oracle's bit for bit.
"""

import numpy as np
import pytest

import oracle
from paper_2506_01986_amd import configs, synth
from tests import ties

pytestmark = pytest.mark.gpu

TOL = {"fp32": (1e-5, 1e-5), "bf16": (1e-2, 2e-2)}


def say(*a):
    print(*a, flush=True)


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible GPU"
    from paper_2506_01986_amd import specmemo
    specmemo.load()
    return torch


def close(gpu, ref, dtype):
    atol, rtol = TOL[dtype]
    err = np.abs(gpu - ref) - (atol + rtol * np.abs(ref))
    return float(err.max()) if err.size else -1.0


def check_topk(cfg, z64, gpu_ids):
    """gpu_ids[b, i] equals the stable descending order of z64[b, i] in its
    first k entries and -1 after them, for every row (the batch has been
    cleared of near-ties, so the order is unambiguous).  Returns the number
    of rows compared exactly."""
    B, nh, _ = z64.shape
    exact = 0
    for b in range(B):
        for i in range(nh):
            k = cfg.topk[i]
            assert not ties.near_tie_heads(cfg, z64[b]), (b, "near-tie left by the guard")
            ref = np.argsort(-z64[b, i], kind="stable")[:k]
            assert gpu_ids[b, i, :k].tolist() == ref.tolist(), (b, i, gpu_ids[b, i, :k], ref)
            assert np.all(gpu_ids[b, i, k:] == -1)
            exact += 1
    return exact


def attn_sample(wl, max_rows, rng, full_longest=0):
    """(node, head) pairs: every row when small, else every row of the
    `full_longest` sequences with the most committed keys (their KV ranges are
    split into the most chunks) plus a sample that covers each sequence's
    root, deepest and last node."""
    cfg = wl.cfg
    total = wl.total_nodes * cfg.n_q
    if total <= max_rows:
        return None
    pairs = set()
    for b in np.argsort(-wl.lens, kind="stable")[:full_longest]:
        o, N = int(wl.node_off[b]), wl.trees[b].n
        pairs.update((n, h) for n in range(o, o + N) for h in range(cfg.n_q))
    max_rows += len(pairs)
    for b in range(cfg.B):
        o, N = int(wl.node_off[b]), wl.trees[b].n
        deep = o + int(np.argmax(wl.trees[b].depth))
        for n in (o, deep, o + N - 1):
            for h in rng.choice(cfg.n_q, size=min(cfg.n_q, 4), replace=False):
                pairs.add((n, int(h)))
    while len(pairs) < max_rows:
        pairs.add((int(rng.integers(wl.total_nodes)), int(rng.integers(cfg.n_q))))
    return np.array(sorted(pairs), dtype=np.int32)


def distinct_sibling_tokens(wl, rng):
    tok = np.zeros(wl.total_nodes, np.int32)
    for b, t in enumerate(wl.trees):
        o = int(wl.node_off[b])
        tok[o] = wl.root_tok[b]
        for u in range(t.n):
            kids = synth.children(t, u)
            if kids:
                tok[o + np.array(kids)] = rng.choice(wl.cfg.vocab, size=len(kids), replace=False)
    return tok


def run_parity(torch, wl, max_attn_rows=None, typical=True, label="", pack_heads=True, full_longest=0):
    from paper_2506_01986_amd import runner, specmemo as sm
    cfg = wl.cfg
    say(f"[parity] {label or cfg.name}: B={cfg.B} sumN={wl.total_nodes} L={wl.lens.tolist()[:8]}")
    rng = np.random.default_rng(1234)
    z64, redrawn = ties.guard_hidden(wl)
    say(f"[parity]   near-tie guard: re-drawn hidden states {redrawn}")
    step = runner.VerifyStep(wl, keep_logits=True, pack_heads=pack_heads)

    # (a) head projection, top-k, tree tokens
    say("[parity]   stage a")
    step.medusa_topk()
    torch.cuda.synchronize()
    z_gpu = step.logits.cpu().numpy()
    ids_gpu = step.topk_ids.cpu().numpy()
    tok_gpu = step.node_tok.cpu().numpy()
    assert close(z_gpu, z64, cfg.dtype) <= 0
    err = np.abs(z_gpu - z64) / (1.0 + np.abs(z64))
    say(f"[parity]   logits: max |z_gpu - z64| / (1 + |z|) = {float(err.max()):.3g} (bound {ties.TIE_REL:g})")
    assert float(err.max()) <= ties.TIE_REL
    exact = check_topk(cfg, z64, ids_gpu)
    # the same decision taken in the kernel's precision: the oracle's top-k over
    # the GPU's own fp32 logits must pick exactly the GPU's ids
    ids32, _ = oracle.heads_topk(z_gpu.astype(np.float64), cfg.topk, cfg.kmax)
    assert np.array_equal(ids_gpu, ids32)
    ids64, _ = oracle.heads_topk(z64, cfg.topk, cfg.kmax)
    tok64 = oracle.tree_tokens(wl.node_off, wl.depth, wl.rank, wl.root_tok, ids64)
    assert np.array_equal(tok_gpu, oracle.tree_tokens(wl.node_off, wl.depth, wl.rank, wl.root_tok, ids_gpu))
    assert np.array_equal(ids_gpu, ids64)
    assert np.array_equal(tok_gpu, tok64)
    assert exact == cfg.B * cfg.n_heads
    if step.head_layout == sm.HEADS_PACKED:
        # the fused form (no logits kept): the projection hands each 64-row
        # group's top-k to the top-k pass; the same ids, values and tree tokens
        vals_gpu = step.topk_vals.cpu().numpy()
        keep, step.logits = step.logits, None
        step.topk_ids.fill_(-7)
        step.node_tok.fill_(-7)
        step.topk_vals.fill_(0)
        step.medusa_topk()
        torch.cuda.synchronize()
        step.logits = keep
        assert np.array_equal(step.topk_ids.cpu().numpy(), ids64)
        assert np.array_equal(step.node_tok.cpu().numpy(), tok64)
        assert np.array_equal(step.topk_vals.cpu().numpy().view(np.uint32), vals_gpu.view(np.uint32))
    say(f"[parity]   stage a ok: exact top-k rows {exact}/{cfg.B * cfg.n_heads}")

    # (b) tree attention
    say("[parity]   stage b")
    step.tree_attn()
    torch.cuda.synchronize()
    out_gpu = runner.to_host_storage(step.out, cfg.dtype)
    out_gpu = synth.storage_to_f64(out_gpu, cfg.dtype)
    sel = attn_sample(wl, max_attn_rows or 10 ** 9, rng, full_longest)
    ref = oracle.tree_attn(wl.q, wl.pool_k, wl.pool_v, wl.node_off, wl.parent, wl.lens, wl.seq_base,
                           cfg.n_kv, sel=sel)
    got = out_gpu if sel is None else out_gpu[sel[:, 0], sel[:, 1]]
    worst = close(got, ref, cfg.dtype)
    say(f"[parity]   stage b rows={ref.shape[0] if sel is not None else ref.shape[0] * ref.shape[1]} "
        f"max|err|={np.abs(got - ref).max():.3g} margin={worst:.3g}")
    assert worst <= 0

    # (c) acceptance on planted logits (oracle node tokens plant the walk)
    lg = synth.planted_logits(wl, tok64)
    step.set_base_logits(lg)
    stride = step.path_stride
    modes = [(sm.GREEDY, "greedy")] + ([(sm.TYPICAL, "typical")] if typical else [])
    for mode, name in modes:
        say(f"[parity]   stage c {name}")
        step.mode = mode
        if mode == sm.TYPICAL:
            need = sm.workspace_bytes(sm.WS_ACCEPT, step.dt, step.trees, None, mode)
            if step.ws.numel() < need:
                step.ws = torch.empty(need, dtype=torch.uint8, device="cuda")
                step.ws_bytes = need
        step.accept()
        torch.cuda.synchronize()
        if mode == sm.GREEDY:
            ra, rp, rn = oracle.accept_greedy(lg, tok64, wl.node_off, wl.parent, wl.depth, stride)
        else:
            ra, rp, rn = oracle.accept_typical(lg, tok64, wl.node_off, wl.parent, wl.depth, stride,
                                               step.temperature, step.eps, step.delta)
        assert np.array_equal(step.accept_len.cpu().numpy(), ra)
        assert np.array_equal(step.path.cpu().numpy(), rp)
        assert np.array_equal(step.next_tok.cpu().numpy(), rn)
        for b in range(cfg.B):
            assert rp[b, :ra[b] + 1].tolist() == wl.plan_path[b]
    step.mode = sm.GREEDY

    # (d) compaction, after a greedy acceptance
    say("[parity]   stage d")
    step.accept()
    K0, V0 = wl.pool_k.copy(), wl.pool_v.copy()
    step.kv_compact()
    torch.cuda.synchronize()
    acc, path = step.accept_len.cpu().numpy(), step.path.cpu().numpy()
    new_len = oracle.kv_compact(K0, V0, wl.seq_base, wl.lens, acc, path)
    Kg = runner.to_host_storage(step.k, cfg.dtype)
    Vg = runner.to_host_storage(step.v, cfg.dtype)
    assert np.array_equal(Kg.view(np.uint8), K0.view(np.uint8))
    assert np.array_equal(Vg.view(np.uint8), V0.view(np.uint8))
    assert np.array_equal(step.seq_len.cpu().numpy(), new_len)
    say(f"[parity]   stage d ok: accepted {acc.tolist()[:10]}")

    # (c) + (d) fused into one call, from the original pool, both modes
    for mode, name in modes:
        say(f"[parity]   stages c+d fused, {name}")
        step.reset_pool()
        step.mode = mode
        step.accept_compact()
        torch.cuda.synchronize()
        if mode == sm.GREEDY:
            ra, rp, rn = oracle.accept_greedy(lg, tok64, wl.node_off, wl.parent, wl.depth, stride)
        else:
            ra, rp, rn = oracle.accept_typical(lg, tok64, wl.node_off, wl.parent, wl.depth, stride,
                                               step.temperature, step.eps, step.delta)
        assert np.array_equal(step.accept_len.cpu().numpy(), ra)
        assert np.array_equal(step.path.cpu().numpy(), rp)
        assert np.array_equal(step.next_tok.cpu().numpy(), rn)
        K0, V0 = wl.pool_k.copy(), wl.pool_v.copy()
        new_len = oracle.kv_compact(K0, V0, wl.seq_base, wl.lens, ra, rp)
        assert np.array_equal(runner.to_host_storage(step.k, cfg.dtype).view(np.uint8), K0.view(np.uint8))
        assert np.array_equal(runner.to_host_storage(step.v, cfg.dtype).view(np.uint8), V0.view(np.uint8))
        assert np.array_equal(step.seq_len.cpu().numpy(), new_len)
    step.mode = sm.GREEDY
    return step


# attention rows compared: every row, or (sampled rows, sequences compared whole)
CONFIG_ROWS = {"tiny_fp32": None, "llama2_7b_b1": None, "llama2_13b_b4": None, "llama2_70b_b10": None,
               "stress_b32": (6000, 4)}


@pytest.mark.parametrize("name", list(CONFIG_ROWS))
def test_config_parity(torch_cuda, name):
    cfg = configs.get(name)
    wl = synth.make(cfg)
    rows, whole = CONFIG_ROWS[name] or (None, 0)
    run_parity(torch_cuda, wl, max_attn_rows=rows, full_longest=whole)


# the same workloads drawn from other seeds (lengths, trees, values, planted walks)
@pytest.mark.parametrize("name,seed", [("llama2_13b_b4", 101), ("llama2_70b_b10", 101), ("llama2_70b_b10", 102),
                                       ("stress_b32", 101)])
def test_config_parity_other_seeds(torch_cuda, name, seed):
    cfg = configs.get(name)
    wl = synth.make(cfg, seed=seed)
    rows, whole = CONFIG_ROWS[name] or (None, 0)
    run_parity(torch_cuda, wl, max_attn_rows=rows, full_longest=whole, label=f"{name} seed {seed}")


def edge_cfg(**kw):
    base = dict(name="edge", dtype="bf16", B=3, n_q=8, n_kv=1, head_dim=128, hidden=136, vocab=1000,
                n_heads=4, topk=(10, 10, 10, 10), tree="T64", kv_len=(1, 1), seed=77, w_std=0.05)
    base.update(kw)
    return configs.Config(**base)


EDGES = {
    # empty committed range, single-node tree, 128-node GQA tree (1024 query rows), ragged short L
    "mixed_gqa": (edge_cfg(B=4, n_q=8, n_kv=1),
                  lambda r: [synth.random_tree(r, 128), synth.tree_from_rank_paths([()]), synth.t64(),
                             synth.chain_tree(5)], [0, 37, 64, 1]),
    # MHA (64-row items: the key-split form), 17 sequences (two 16-wide batch tiles in the head GEMM)
    "mha_b17": (edge_cfg(B=17, n_q=2, n_kv=2, hidden=64, vocab=520),
                lambda r: [synth.random_tree(r, int(r.integers(1, 65))) for _ in range(17)],
                list(range(0, 17 * 70, 70))),
    # more than 32 sequences: one launch with the descriptors in the workspace
    "b40": (edge_cfg(B=40, n_q=4, n_kv=2, hidden=32, vocab=256, topk=(4, 3, 2, 2)),
            lambda r: [synth.random_tree(r, int(r.integers(1, 20)), max_kids=2) for _ in range(40)],
            [int(x) for x in np.random.default_rng(5).integers(0, 300, 40)]),
    # one long sequence alone: the KV range is split into chunks and merged
    "split_kv": (edge_cfg(B=1, n_q=1, n_kv=1, hidden=64, vocab=300),
                 lambda r: [synth.t64()], [20011]),
    # fp32 with GQA and head_dim 64
    "fp32_gqa": (edge_cfg(dtype="fp32", B=3, n_q=6, n_kv=2, head_dim=64, hidden=40, vocab=333, w_std=1.0),
                 lambda r: [synth.t16(), synth.random_tree(r, 30), synth.tree_from_rank_paths([()])],
                 [5, 0, 200]),
    # the deepest trees: 15 heads (paths of 16 nodes), binary branching
    "deep15": (edge_cfg(B=3, n_q=4, n_kv=2, hidden=32, vocab=64, n_heads=15, topk=(2,) * 15, p_accept=0.85),
               lambda r: [synth.chain_tree(16), synth.random_tree(r, 60, max_depth=15, max_kids=2),
                          synth.random_tree(r, 128, max_depth=15, max_kids=2)], [3, 50, 0]),
    # the widest top-k (32 per head) and a 32-child root
    "topk32": (edge_cfg(B=2, n_q=2, n_kv=1, hidden=64, vocab=100, n_heads=2, topk=(32, 32)),
               lambda r: [synth.random_tree(r, 128, max_depth=2, max_kids=32), synth.star_tree(33)], [10, 300]),
    # multi-query attention: 64 query heads on one KV head, 8192 query rows per sequence
    "mqa64": (edge_cfg(B=2, n_q=64, n_kv=1, hidden=64, vocab=300),
              lambda r: [synth.random_tree(r, 128), synth.t16()], [300, 2000]),
    # more than 32 sequences, some long enough to split: one launch (descriptor table in the workspace)
    "b36_split": (edge_cfg(B=36, n_q=8, n_kv=2, hidden=32, vocab=256),
                  lambda r: [synth.random_tree(r, int(r.integers(1, 65))) for _ in range(36)],
                  [5000, 3000] + [int(x) for x in np.random.default_rng(7).integers(0, 1500, 34)]),
    # the largest batch (4096 sequences, one launch per stage), the smallest hidden size
    "b4096": (edge_cfg(B=4096, n_q=1, n_kv=1, hidden=8, vocab=16, n_heads=1, topk=(4,)),
              lambda r: [synth.random_tree(r, int(r.integers(1, 6)), max_depth=1, max_kids=4) for _ in range(4096)],
              [int(x) for x in np.random.default_rng(6).integers(0, 31, 4096)]),
}


# edge cases whose heads stay in the row-major (nn.Linear) layout; the others
# use the packed layout, as do the five workloads
ROWMAJOR_HEADS = {"mha_b17", "split_kv"}


@pytest.mark.parametrize("name", list(EDGES))
def test_edge_parity(torch_cuda, name):
    cfg, trees, lens = EDGES[name]
    rng = np.random.default_rng(len(name))
    wl = synth.make(cfg, trees=trees(rng), lens=lens)
    run_parity(torch_cuda, wl, label=name, pack_heads=name not in ROWMAJOR_HEADS)


def test_budgeted_tree_sizes(torch_cuda):
    """Tree sizes chosen from each slab's free rows: a 128-node default tree
    (depth 4, top-10) pruned right to left to what the slab still holds, full
    slabs sitting the step out, every other slab filled to the last row.  The
    library's builder and planner must give the oracle's trees, which then go
    through the whole step."""
    from oracle import budget as ob
    from paper_2506_01986_amd import specmemo as sm
    rng = np.random.default_rng(21)
    default = ob.build_tree(128, 45, 4, 10)
    assert [list(map(int, a)) for a in sm.tree_build(128, 45, 4, 10)] == [list(a) for a in default]
    free = [0, 1, 2, 3, 7, 16, 33, 64, 100, 127, 128, 129, 500]
    lens = [int(x) for x in rng.integers(0, 3000, len(free))]
    caps = [n + f for n, f in zip(lens, free)]
    sizes = ob.plan_tree_sizes(lens, caps, 128)
    assert list(map(int, sm.plan_tree_sizes(lens, caps, 128))) == sizes
    run = [b for b in range(len(free)) if sizes[b] > 0]
    trees = [synth.Tree(*(np.asarray(a[:sizes[b]], np.int32) for a in default)) for b in run]
    cfg = edge_cfg(B=len(run), n_q=8, n_kv=2, hidden=64, vocab=700, seed=21)
    wl = synth.make(cfg, trees=trees, lens=[lens[b] for b in run], caps=[caps[b] for b in run])
    say(f"[parity] budgeted sizes {[sizes[b] for b in run]}")
    run_parity(torch_cuda, wl, label="budgeted_tree_sizes")


def test_topk_ties(torch_cuda):
    """Integer-valued heads and hidden states give exact fp32 logits with many
    ties: head 0 is all zeros (every logit ties; the candidate buffer
    overflows), head 1 has entries in {-1, 0, 1}, head 2 is Gaussian, head 3
    puts a few large values over a flat floor.  Ids must equal the oracle's
    exactly (equal values by lower id), for both head layouts."""
    from paper_2506_01986_amd import runner
    cfg = edge_cfg(B=3, n_q=8, n_kv=1, hidden=64, vocab=5000, topk=(10, 10, 10, 10), seed=5)
    wl = synth.make(cfg, trees=[synth.t64()] * 3, lens=[10, 20, 30])
    rng = np.random.default_rng(5)
    w = np.zeros((4, cfg.vocab, cfg.hidden), np.float32)
    w[1] = rng.integers(-1, 2, size=(cfg.vocab, cfg.hidden))
    w[2] = np.round(rng.standard_normal((cfg.vocab, cfg.hidden)) * 4)
    w[3] = -1.0
    w[3, rng.choice(cfg.vocab, 40, replace=False)] = 3.0
    h = rng.integers(-1, 2, size=(cfg.B, cfg.hidden)).astype(np.float32)
    h[:, 0] = 1.0
    wl.head_w = synth.to_bf16_bits(w)
    wl.hidden = synth.to_bf16_bits(h)
    z64 = oracle.head_logits(wl.hidden, wl.head_w)
    ids64, _ = oracle.heads_topk(z64, cfg.topk, cfg.kmax)
    for pack, keep in ((True, True), (False, True), (True, False)):   # (True, False): the fused form
        step = runner.VerifyStep(wl, keep_logits=keep, pack_heads=pack)
        step.medusa_topk()
        torch_cuda.cuda.synchronize()
        if keep:
            assert np.array_equal(step.logits.cpu().numpy(), z64.astype(np.float32))
        assert np.array_equal(step.topk_ids.cpu().numpy(), ids64), (pack, keep)
        assert np.array_equal(step.topk_ids.cpu().numpy()[:, 0], np.tile(np.arange(10), (3, 1)))


def test_pack_heads_layout(torch_cuda):
    """The packed buffer holds head_w[i][64 G + 16 t + l % 16][32 s + 8 (l / 16) + e]
    at element ((((i nG + G) nS + s) 4 + t) 64 + l) 8 + e, zero past vocab and hidden."""
    import torch
    from paper_2506_01986_amd import specmemo as sm
    n_heads, vocab, hidden = 2, 150, 72          # ragged in both row groups and k steps
    rng = np.random.default_rng(9)
    w = rng.integers(1, 0x7F00, size=(n_heads, vocab, hidden)).astype(np.uint16)   # distinct-ish bit patterns
    src = torch.from_numpy(w.view(np.int16)).cuda()
    nbytes = sm.packed_heads_bytes(sm.BF16, n_heads, vocab, hidden)
    nG, nS = -(-vocab // 64), -(-hidden // 32)
    assert nbytes == n_heads * nG * nS * 4096
    dst = torch.full((nbytes // 2,), -1, dtype=torch.int16, device="cuda")
    sm.pack_heads(sm.BF16, n_heads, vocab, hidden, src, dst)
    got = dst.cpu().numpy().view(np.uint16)
    want = np.zeros(nbytes // 2, np.uint16)
    for i in range(n_heads):
        for G in range(nG):
            for s in range(nS):
                for t in range(4):
                    for l in range(64):
                        row, col = 64 * G + 16 * t + l % 16, 32 * s + 8 * (l // 16)
                        if row < vocab and col < hidden:
                            o = ((((i * nG + G) * nS + s) * 4 + t) * 64 + l) * 8
                            want[o:o + 8] = w[i, row, col:col + 8]
    assert np.array_equal(got, want)


def test_acceptance_small_vocab_random(torch_cuda):
    """Random tiny trees and logits with many ties: greedy and typical vs oracle."""
    import torch
    from paper_2506_01986_amd import specmemo as sm
    rng = np.random.default_rng(3)
    trees = [synth.random_tree(rng, int(rng.integers(1, 13)), max_depth=4, max_kids=4) for _ in range(64)]
    vocab = 8
    node_off = np.concatenate([[0], np.cumsum([t.n for t in trees])]).astype(np.int32)
    parent = np.concatenate([t.parent for t in trees])
    depth = np.concatenate([t.depth for t in trees])
    rank = np.concatenate([t.rank for t in trees])
    tok = np.zeros(node_off[-1], np.int32)
    for b, t in enumerate(trees):
        for u in range(t.n):
            kids = synth.children(t, u)
            if kids:
                tok[node_off[b] + np.array(kids)] = rng.choice(vocab, size=len(kids), replace=False)
    tr = sm.Trees(node_off, parent, depth, rank, device="cuda")
    B, stride = len(trees), 5
    for dtype in ("fp32", "bf16"):
        raw = rng.integers(0, 3, size=(node_off[-1], vocab)).astype(np.float32)
        raw[::3] = (2 * rng.standard_normal((len(raw[::3]), vocab))).astype(np.float32)
        lg = raw if dtype == "fp32" else synth.to_bf16_bits(raw)
        from paper_2506_01986_amd.runner import to_device
        dlg = to_device(lg, dtype, "cuda")
        dtok = torch.from_numpy(tok).cuda()
        out = [torch.empty(B, dtype=torch.int32, device="cuda"), torch.empty((B, stride), dtype=torch.int32, device="cuda"),
               torch.empty(B, dtype=torch.int32, device="cuda")]
        dt = sm.FP32 if dtype == "fp32" else sm.BF16
        wsg = torch.empty(sm.workspace_bytes(sm.WS_ACCEPT, dt, tr, None, sm.GREEDY), dtype=torch.uint8, device="cuda")
        sm.accept(dt, tr, vocab, sm.GREEDY, dlg, dtok, out[0], out[1], stride, out[2], ws=wsg, ws_bytes=wsg.numel())
        ra, rp, rn = oracle.accept_greedy(lg, tok, node_off, parent, depth, stride)
        assert np.array_equal(out[0].cpu().numpy(), ra)
        assert np.array_equal(out[1].cpu().numpy(), rp)
        assert np.array_equal(out[2].cpu().numpy(), rn)
        # typical: compare where no edge that can matter sits within fp32 error of its threshold
        ws = torch.empty(sm.workspace_bytes(sm.WS_ACCEPT, dt, tr, None, sm.TYPICAL), dtype=torch.uint8, device="cuda")
        sm.accept(dt, tr, vocab, sm.TYPICAL, dlg, dtok, out[0], out[1], stride, out[2], temperature=0.7,
                  eps=0.09, delta=0.3, ws=ws, ws_bytes=ws.numel())
        ra, rp, rn, lp, lt = oracle.accept_typical(lg, tok, node_off, parent, depth, stride, 0.7, 0.09, 0.3,
                                                   edges=True)
        ga, gp, gn = (o.cpu().numpy() for o in out)
        checked = 0
        for b in range(B):
            o, n1 = node_off[b], node_off[b + 1]
            margin = np.abs(lp[o + 1:n1] - lt[o + 1:n1])
            if margin.size and margin.min() < 1e-4:
                continue
            checked += 1
            assert ga[b] == ra[b] and np.array_equal(gp[b], rp[b]) and gn[b] == rn[b], b
        assert checked > B // 2


def _typical_rows(rng, trees, vocab, dtype, T, eps, delta):
    """Unplanted N(0, 1) logit rows for typical acceptance, with distinct
    sibling tokens; along one walk per tree the chosen child's token is
    placed just above its edge threshold and one sibling's just below, at
    margins of 2e-4 .. 0.2 in log-probability (fp32 keeps them; bf16 rounds
    them to its grid).  The placement reads the oracle's row statistics."""
    node_off = np.concatenate([[0], np.cumsum([t.n for t in trees])]).astype(np.int32)
    N = int(node_off[-1])
    z = rng.standard_normal((N, vocab)).astype(np.float32)
    tok = np.zeros(N, np.int32)
    placed = []                                   # (row u, token, margin)
    margins = [2e-4, 5e-4, 1e-3, 3e-3, 0.02, 0.2]
    for b, t in enumerate(trees):
        o = int(node_off[b])
        for u in range(t.n):
            kids = synth.children(t, u)
            if kids:
                tok[o + np.array(kids)] = rng.choice(vocab, size=len(kids), replace=False)
        u = 0
        while synth.children(t, u):
            kids = synth.children(t, u)
            c = kids[int(rng.integers(len(kids)))]
            m = float(rng.choice(margins))
            placed.append((o + u, int(tok[o + c]), m))
            if len(kids) > 1:
                sib = next(k for k in kids if k != c)
                placed.append((o + u, int(tok[o + sib]), -float(rng.choice(margins))))
            u = c
    for _ in range(4):                            # lse and H move slightly with each placed value
        lse, H = oracle.softmax_stats(z, T)
        for u, v, m in placed:
            lthr = min(np.log(eps), np.log(delta) - H[u])
            z[u, v] = np.float32(T * (lthr + m + lse[u]))
    return (z if dtype == "fp32" else synth.to_bf16_bits(z)), tok, node_off


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_typical_full_vocab(torch_cuda, dtype):
    """Typical acceptance (App. A.1) at the 70B-shaped batch's size: ten
    64-node trees, vocabulary 32000, unplanted rows.  The per-row statistics
    the kernel leaves in the workspace (lse and entropy of softmax(z / T))
    must match the oracle's, and the accepted lengths, paths and next tokens
    must be bit-exact for every sequence whose edges all lie more than 1e-4
    (log units) from their thresholds (the guard of the fp32 decision)."""
    import torch
    from paper_2506_01986_amd import specmemo as sm
    from paper_2506_01986_amd.runner import to_device
    T, eps, delta = 0.7, 0.09, 0.3
    rng = np.random.default_rng(70)
    trees = [synth.t64() for _ in range(10)]
    lg, tok, node_off = _typical_rows(rng, trees, 32000, dtype, T, eps, delta)
    parent = np.concatenate([t.parent for t in trees])
    depth = np.concatenate([t.depth for t in trees])
    rank = np.concatenate([t.rank for t in trees])
    tr = sm.Trees(node_off, parent, depth, rank, device="cuda")
    B, N, stride = len(trees), int(node_off[-1]), 5
    dt = sm.FP32 if dtype == "fp32" else sm.BF16
    ws = torch.empty(sm.workspace_bytes(sm.WS_ACCEPT, dt, tr, None, sm.TYPICAL), dtype=torch.uint8, device="cuda")
    out = [torch.full((B,), -7, dtype=torch.int32, device="cuda"),
           torch.full((B, stride), -7, dtype=torch.int32, device="cuda"),
           torch.full((B,), -7, dtype=torch.int32, device="cuda")]
    say(f"[typical] {dtype}: B={B} rows={N} vocab=32000")
    sm.accept(dt, tr, 32000, sm.TYPICAL, to_device(lg, dtype, "cuda"), torch.from_numpy(tok).cuda(), out[0], out[1],
              stride, out[2], temperature=T, eps=eps, delta=delta, ws=ws, ws_bytes=ws.numel())
    torch.cuda.synchronize()
    stats = ws[:8 * N].view(torch.float32).cpu().numpy().reshape(N, 2).astype(np.float64)
    lse, H = oracle.softmax_stats(lg, T)
    e_lse, e_H = np.abs(stats[:, 0] - lse).max(), np.abs(stats[:, 1] - H).max()
    say(f"[typical]   max |lse err| {e_lse:.3g}, max |H err| {e_H:.3g}, H in [{H.min():.3f}, {H.max():.3f}]")
    assert e_lse <= 2e-5 and e_H <= 2e-5               # fp32 sums over 32000 terms: a few 1e-6
    ra, rp, rn, lp, lt = oracle.accept_typical(lg, tok, node_off, parent, depth, stride, T, eps, delta, edges=True)
    ga, gp, gn = (o.cpu().numpy() for o in out)
    checked = 0
    for b in range(B):
        o, n1 = node_off[b], node_off[b + 1]
        if np.abs(lp[o + 1:n1] - lt[o + 1:n1]).min() < 1e-4:
            continue
        checked += 1
        assert ga[b] == ra[b] and np.array_equal(gp[b], rp[b]) and gn[b] == rn[b], (b, ga[b], ra[b])
    margins = np.abs(lp - lt)[np.isfinite(lp)]
    say(f"[typical]   accepted {(ra + 1).tolist()}, compared {checked}/{B}, smallest edge margin {margins.min():.2g}")
    assert checked == B
    assert ra.max() >= 2                          # the placed walks reach past the first level


def _argbest_rows(rng, vocab, n):
    """Logit rows (float32, exactly representable in bf16) that stress the arg-best order."""
    rows = []
    for r in range(n):
        kind = r % 8
        x = rng.standard_normal(vocab).astype(np.float32)
        x = np.float32(synth.storage_to_f64(synth.to_bf16_bits(x), "bf16"))   # bf16 grid: ties at the max are common
        if kind == 1:
            x[-1] = 50.0                                   # max at the last id
        elif kind == 2:
            x[0] = 50.0                                    # max at the first id
        elif kind == 3:
            x[:] = 1.5                                     # all equal: id 0
        elif kind == 4:
            x = -np.abs(x) - 1.0
            i, j = sorted(rng.choice(vocab, 2, replace=False))
            x[i], x[j] = -0.0, 0.0                         # -0 first, +0 later: equal, lower id wins
        elif kind == 5:
            x = -np.abs(x) - 1.0
            i, j = sorted(rng.choice(vocab, 2, replace=False))
            x[i], x[j] = 0.0, -0.0
        elif kind == 6:
            x[:] = -np.inf                                 # all -inf: id 0
        elif kind == 7:
            top = x.max()
            x[rng.choice(vocab, 5, replace=False)] = top   # several ties at the max
        rows.append(x)
    return np.stack(rows)


@pytest.mark.parametrize("vocab", [8, 1000, 1004, 32000, 32768, 32776])
def test_greedy_argbest_rows(torch_cuda, vocab):
    """Single-node trees: next_tok is each row's arg-best (larger value, then lower id; -0 == +0)."""
    import torch
    from paper_2506_01986_amd import specmemo as sm
    from paper_2506_01986_amd.runner import to_device
    rng = np.random.default_rng(vocab)
    B, stride = 48, 5
    node_off = np.arange(B + 1, dtype=np.int32)
    zeros = np.zeros(B, np.int32)
    tr = sm.Trees(node_off, np.full(B, -1, np.int32), zeros, zeros, device="cuda")
    raw = _argbest_rows(rng, vocab, B)
    tok = torch.zeros(B, dtype=torch.int32, device="cuda")
    for dtype in ("bf16", "fp32"):
        say(f"argbest vocab={vocab} {dtype}")
        lg = raw if dtype == "fp32" else synth.to_bf16_bits(raw)
        dt = sm.FP32 if dtype == "fp32" else sm.BF16
        dlg = to_device(lg, dtype, "cuda")
        acc = torch.empty(B, dtype=torch.int32, device="cuda")
        path = torch.empty((B, stride), dtype=torch.int32, device="cuda")
        nxt = torch.empty(B, dtype=torch.int32, device="cuda")
        ws = torch.empty(sm.workspace_bytes(sm.WS_ACCEPT, dt, tr, None, sm.GREEDY), dtype=torch.uint8, device="cuda")
        sm.accept(dt, tr, vocab, sm.GREEDY, dlg, tok, acc, path, stride, nxt, ws=ws, ws_bytes=ws.numel())
        ra, rp, rn = oracle.accept_greedy(lg, np.zeros(B, np.int32), node_off, np.full(B, -1, np.int32), zeros, stride)
        assert np.array_equal(nxt.cpu().numpy(), rn)
        assert np.array_equal(acc.cpu().numpy(), ra) and np.array_equal(path.cpu().numpy(), rp)


@pytest.mark.parametrize("fused", [False, True, "overlapped"], ids=["four_calls", "accept_compact", "overlapped"])
def test_graph_replay(torch_cuda, fused):
    """The calls of a step (four, or three with acceptance and compaction
    fused) captured in one HIP graph.  Every replay, with eager work between
    replays (the pool restored, every output poisoned), reproduces the eager
    step bit for bit: no call records a memset, an allocation or a host
    synchronisation, and the kernels read nothing that capture freezes except
    their arguments."""
    import torch
    from paper_2506_01986_amd import runner
    rng = np.random.default_rng(21)
    cfg = edge_cfg(B=5, n_q=8, n_kv=2, hidden=256, vocab=3000, seed=21)
    trees = [synth.t64(), synth.t16(), synth.random_tree(rng, 40), synth.chain_tree(5), synth.random_tree(rng, 100)]
    wl = synth.make(cfg, trees=trees, lens=[900, 0, 300, 2500, 64])
    step = runner.VerifyStep(wl)
    step.medusa_topk()
    torch.cuda.synchronize()
    step.set_base_logits(synth.planted_logits(wl, step.node_tok.cpu().numpy()))
    k0, v0, len0 = step.k.clone(), step.v.clone(), step.seq_len.clone()
    outs = [step.topk_ids, step.node_tok, step.out, step.accept_len, step.path, step.next_tok, step.seq_len,
            step.k, step.v]

    def restore_and_poison():
        step.k.copy_(k0)
        step.v.copy_(v0)
        step.seq_len.copy_(len0)
        for t in (step.topk_ids, step.node_tok, step.accept_len, step.path, step.next_tok):
            t.fill_(-7)
        step.out.zero_()

    run = step.run_overlapped if fused == "overlapped" else step.run_fused if fused else step.run
    restore_and_poison()
    step.run_fused() if fused == "overlapped" else run()    # the overlapped step must equal the serial one
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]
    if fused == "overlapped":
        for r in range(3):
            restore_and_poison()
            run()
            torch.cuda.synchronize()
            for i, (a, b) in enumerate(zip(ref, outs)):
                assert torch.equal(a.contiguous().view(torch.uint8), b.contiguous().view(torch.uint8)), ("eager", r, i)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    torch.cuda.synchronize()
    for r in range(3):
        say(f"graph replay {r}")
        restore_and_poison()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(ref, outs)):   # bits: the pool's canary rows hold NaN patterns
            assert torch.equal(a.contiguous().view(torch.uint8), b.contiguous().view(torch.uint8)), (r, i)


def test_run_to_run_determinism(torch_cuda):
    import torch
    from paper_2506_01986_amd import runner
    cfg, trees, lens = EDGES["split_kv"]
    wl = synth.make(cfg, trees=trees(np.random.default_rng(0)), lens=lens)
    step = runner.VerifyStep(wl, keep_logits=True)
    outs = []
    for _ in range(2):
        step.medusa_topk()
        step.tree_attn()
        torch.cuda.synchronize()
        outs.append((step.logits.clone(), step.out.clone(), step.topk_ids.clone()))
    for a, b in zip(*outs):
        assert torch.equal(a.view(torch.uint8) if a.dtype != torch.int32 else a,
                           b.view(torch.uint8) if b.dtype != torch.int32 else b)


@pytest.mark.parametrize("env,many", [({"SPECMEMO_ATTN_ROWS": "64"}, False), ({"SPECMEMO_ATTN_ROWS": "256"}, False),
                                      ({"SPECMEMO_ATTN_XCD": "0"}, False), ({"SPECMEMO_ATTN_CHUNK": "256"}, False),
                                      ({"SPECMEMO_ATTN_CHUNK": "0"}, False), ({}, True),
                                      ({"SPECMEMO_ATTN_XCD": "0"}, True), ({"SPECMEMO_ATTN_CHUNK": "256"}, True)],
                         ids=["rows64", "rows256", "no_xcd_order", "chunk256", "no_split", "b40_table",
                              "b40_table_no_xcd_order", "b40_table_chunk256"])
def test_attention_tuning_overrides(torch_cuda, env, many):
    """The attention's tuning variables (read once per process) change the
    work split, not the result: each runs in a child process of its own,
    one after the other, against the oracle."""
    import os
    import subprocess
    import sys
    child = os.path.join(os.path.dirname(os.path.abspath(__file__)), "attn_override_check.py")
    say(f"[override] {env}")
    r = subprocess.run([sys.executable, child] + (["many"] if many else []), env={**os.environ, **env},
                       capture_output=True, text=True, timeout=240)
    say(r.stdout.strip())
    assert r.returncode == 0, r.stdout + r.stderr[-3000:]
