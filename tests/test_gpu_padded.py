"""GPU parity of the padded-batching variant (Sec. 3.3, Fig. 8) against the
oracle: attention over a cache holding pad tokens (-inf in the mask), and the
padded KV update (accepted rows moved, pad rows flagged, positions skipping
pads).  Floats within the bf16 / fp32 tolerances of the ragged path, integers,
flags and moved rows bit-exact."""

import numpy as np
import pytest

import oracle
from oracle import padded as opad
from paper_2506_01986_amd import configs, synth

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
    return float((np.abs(gpu - ref) - (atol + rtol * np.abs(ref))).max())


def edge_cfg(**kw):
    base = dict(name="edge", dtype="bf16", B=3, n_q=8, n_kv=1, head_dim=128, hidden=136, vocab=1000,
                n_heads=4, topk=(10, 10, 10, 10), tree="T64", kv_len=(1, 1), seed=77, w_std=0.05)
    base.update(kw)
    return configs.Config(**base)


def padded_workload(cfg, trees, real_lens, steps, seed, pad_runs=None):
    rng = np.random.default_rng(seed)
    rows, slab = synth.padded_history(rng, real_lens, steps, 0.6, cfg.n_heads)
    for b, (start, stop) in (pad_runs or {}).items():      # extra runs of pads (whole chunks)
        slab[b][start:stop] = 0
    wl = synth.make(cfg, trees=trees, lens=rows, caps=[int(r) + t.n + 8 for r, t in zip(rows, trees)],
                    with_heads=False)
    return wl, synth.pool_key_flags(wl, slab)


def node_tokens(wl):
    """Seeded tree tokens (the heads' stage is not under test here): the root's
    token, else a function of (depth, rank), so that siblings differ."""
    tok = np.empty(wl.total_nodes, np.int32)
    for b in range(wl.cfg.B):
        o, n = int(wl.node_off[b]), wl.trees[b].n
        d, r = wl.depth[o:o + n].astype(np.int64), wl.rank[o:o + n].astype(np.int64)
        tok[o:o + n] = (97 * d + 13 * r + 5 + b) % wl.cfg.vocab
        tok[o] = wl.root_tok[b]
    return tok


def run_padded_parity(torch, wl, flags, max_rows=None, label=""):
    from paper_2506_01986_amd import runner, specmemo as sm
    cfg = wl.cfg
    say(f"[padded] {label}: B={cfg.B} sumN={wl.total_nodes} L={wl.lens.tolist()[:8]} "
        f"pads={int(sum((flags[int(wl.seq_base[b]):int(wl.seq_base[b]) + int(wl.lens[b])] == 0).sum() for b in range(cfg.B)))}")
    step = runner.VerifyStep(wl, key_valid=flags)
    tok = node_tokens(wl)
    step.node_tok.copy_(torch.from_numpy(tok))

    # attention over the cache with pad tokens
    step.tree_attn_padded()
    torch.cuda.synchronize()
    out = synth.storage_to_f64(runner.to_host_storage(step.out, cfg.dtype), cfg.dtype)
    rng = np.random.default_rng(3)
    total = wl.total_nodes * cfg.n_q
    if max_rows is None or total <= max_rows:
        sel = None
    else:
        flat = rng.choice(total, size=max_rows, replace=False)
        sel = np.stack([flat // cfg.n_q, flat % cfg.n_q], axis=1).astype(np.int32)
    ref = oracle.tree_attn(wl.q, wl.pool_k, wl.pool_v, wl.node_off, wl.parent, wl.lens, wl.seq_base, cfg.n_kv,
                           sel=sel, key_valid=flags)
    got = out if sel is None else out[sel[:, 0], sel[:, 1]]
    margin = close(got, ref, cfg.dtype)
    say(f"[padded]   attention max|err|={np.abs(got - ref).max():.3g} margin={margin:.3g}")
    assert margin <= 0
    # the pads matter: the same rows without the mask differ
    plain = oracle.tree_attn(wl.q, wl.pool_k, wl.pool_v, wl.node_off, wl.parent, wl.lens, wl.seq_base, cfg.n_kv,
                             sel=sel)
    assert close(got, plain, cfg.dtype) > 0

    # greedy acceptance on planted logits, then the padded update
    lg = synth.planted_logits(wl, tok)
    step.set_base_logits(lg)
    step.accept()
    torch.cuda.synchronize()
    acc, path = step.accept_len.cpu().numpy(), step.path.cpu().numpy()
    ra, rp, _ = oracle.accept_greedy(lg, tok, wl.node_off, wl.parent, wl.depth, step.path_stride)
    assert np.array_equal(acc, ra) and np.array_equal(path, rp)
    pos0 = step.pos.cpu().numpy()
    K, V, F = wl.pool_k.copy(), wl.pool_v.copy(), flags.copy()
    new_len, new_pos = opad.pad_update(K, V, wl.seq_base, wl.lens, pos0, F, acc, path)
    step.kv_pad_update()
    torch.cuda.synchronize()
    assert np.array_equal(runner.to_host_storage(step.k, cfg.dtype).view(np.uint8), K.view(np.uint8))
    assert np.array_equal(runner.to_host_storage(step.v, cfg.dtype).view(np.uint8), V.view(np.uint8))
    assert np.array_equal(step.seq_len.cpu().numpy(), new_len)
    assert np.array_equal(step.pos.cpu().numpy(), new_pos)
    words = step.key_valid.cpu().numpy().view(np.uint32)
    assert np.array_equal(sm.unpack_key_valid(words, wl.cap_total), F)
    say(f"[padded]   update ok: accepted {(acc + 1).tolist()[:10]} uniform {int((new_len - wl.lens).max())}")
    return step


PADDED = {
    # GQA, several tree shapes, short prompts
    "mixed": (edge_cfg(B=4, n_q=8, n_kv=2),
              lambda r: [synth.t64(), synth.random_tree(r, 37), synth.t16(), synth.chain_tree(5)],
              [300, 41, 700, 25], 8, None),
    # one long sequence split along its KV range, a whole chunk of pads
    "split_kv": (edge_cfg(B=1, n_q=1, n_kv=1, hidden=64, vocab=300), lambda r: [synth.t64()],
                 [15000], 300, {0: (3000, 9000)}),
    # fp32 path
    "fp32": (edge_cfg(dtype="fp32", B=3, n_q=6, n_kv=2, head_dim=64, hidden=40, vocab=333, w_std=1.0),
             lambda r: [synth.t16(), synth.random_tree(r, 30, max_depth=3), synth.t16()], [90, 30, 200], 10, None),
    # every committed row a pad but the prompt's first
    "mostly_pads": (edge_cfg(B=2, n_q=4, n_kv=1), lambda r: [synth.t16(), synth.t64()], [40, 60], 12,
                    {0: (1, 10 ** 6), 1: (1, 10 ** 6)}),
    # the same with one query head per KV head (64-row items: the key-split form, where one key group
    # of a row can see nothing but pads)
    "mha_mostly_pads": (edge_cfg(B=2, n_q=2, n_kv=2), lambda r: [synth.t16(), synth.t64()], [40, 60], 12,
                        {0: (1, 10 ** 6), 1: (1, 10 ** 6)}),
}


@pytest.mark.parametrize("name", list(PADDED))
def test_padded_parity(torch_cuda, name):
    cfg, trees, lens, steps, runs = PADDED[name]
    rng = np.random.default_rng(len(name))
    t = trees(rng)
    wl, flags = padded_workload(cfg, t, lens, steps, seed=len(name), pad_runs=runs)
    run_padded_parity(torch_cuda, wl, flags, label=name)


def test_padded_parity_70b_shape(torch_cuda):
    """The Llama-2-70B-shaped batch of 10 after 150 padded decode steps (its
    real token counts are the workload's KV lengths), sampled rows."""
    cfg = configs.get("llama2_70b_b10")
    real = synth.make(cfg, with_heads=False).lens
    rng = np.random.default_rng(70)
    rows, slab = synth.padded_history(rng, real, 150, 0.6, cfg.n_heads)
    wl = synth.make(cfg, lens=rows, with_heads=False)
    flags = synth.pool_key_flags(wl, slab)
    run_padded_parity(torch_cuda, wl, flags, max_rows=3000, label="llama2_70b_b10 padded")


def test_padded_update_skips_invalid_paths(torch_cuda):
    """A sequence whose path is not a root path (or whose length is out of
    range) is left untouched and does not set the uniform length."""
    import torch
    from paper_2506_01986_amd import runner
    cfg = edge_cfg(B=3, n_q=2, n_kv=2)
    trees = [synth.t64(), synth.t64(), synth.t16()]
    wl, flags = padded_workload(cfg, trees, [50, 60, 70], 5, seed=4)
    step = runner.VerifyStep(wl, key_valid=flags)
    stride = step.path_stride
    acc = np.array([1, 4, 2], np.int32)
    path = np.full((3, stride), -1, np.int32)
    path[0, :2] = [0, 3]                     # a root path: node 3 is a child of the root
    path[1, :5] = [0, 1, 2, 3, 4]            # increasing, but not a root path (2 is not a child of 1)
    path[2, :3] = [0, 1, 5]                  # a root path of the 16-node tree (5 is a child of 1)
    t16 = synth.t16()
    assert t16.parent[5] == 1 and wl.trees[0].parent[3] == 0 and wl.trees[1].parent[2] != 1
    step.accept_len.copy_(torch.from_numpy(acc))
    step.path.copy_(torch.from_numpy(path))
    pos0 = step.pos.cpu().numpy()
    K, V, F = wl.pool_k.copy(), wl.pool_v.copy(), flags.copy()
    keep = [0, 2]
    new_len, new_pos = opad.pad_update(K, V, wl.seq_base[keep], wl.lens[keep], pos0[keep], F, acc[keep], path[keep])
    step.kv_pad_update()
    torch.cuda.synchronize()
    assert np.array_equal(runner.to_host_storage(step.k, cfg.dtype).view(np.uint8), K.view(np.uint8))
    assert np.array_equal(runner.to_host_storage(step.v, cfg.dtype).view(np.uint8), V.view(np.uint8))
    sl, ps = step.seq_len.cpu().numpy(), step.pos.cpu().numpy()
    assert sl[keep].tolist() == new_len.tolist() and ps[keep].tolist() == new_pos.tolist()
    assert sl[1] == wl.lens[1] and ps[1] == pos0[1]
    from paper_2506_01986_amd import specmemo as sm
    assert np.array_equal(sm.unpack_key_valid(step.key_valid.cpu().numpy().view(np.uint32), wl.cap_total), F)
