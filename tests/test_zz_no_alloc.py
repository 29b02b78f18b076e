"""The allocation-free attention entry point (specmemo_tree_attn_noalloc)
through the C ABI against the workspace form (specmemo_tree_attn) and the
oracle: two calls in a row, the second on a smaller batch, both with split KV
ranges (the partial results live in the library's static scratch)."""

import numpy as np
import pytest

import oracle
from paper_2506_01986_amd import configs, synth

pytestmark = pytest.mark.gpu

TOL = {"fp32": (1e-5, 1e-5), "bf16": (1e-2, 2e-2)}


def say(*a):
    print(*a, flush=True)


def _attn_case(wl):
    import torch
    from paper_2506_01986_amd import runner, specmemo as sm
    cfg = wl.cfg
    dt = sm.BF16 if cfg.dtype == "bf16" else sm.FP32
    trees = sm.Trees(wl.node_off, wl.parent, wl.depth, wl.rank, device="cuda")
    k = runner.to_device(wl.pool_k, cfg.dtype, "cuda")
    v = runner.to_device(wl.pool_v, cfg.dtype, "cuda")
    kv = sm.KVPool(k, v, torch.from_numpy(wl.lens.copy()).cuda(), wl.seq_base, wl.seq_cap, wl.lens)
    q = runner.to_device(wl.q, cfg.dtype, "cuda")
    return sm, runner, dt, trees, kv, q


def _run_both(torch, wl):
    sm, runner, dt, trees, kv, q = _attn_case(wl)
    cfg = wl.cfg
    need = sm.workspace_bytes(sm.WS_ATTN, dt, trees, kv, cfg.n_q)
    assert 0 < need <= sm.STATIC_SCRATCH_BYTES, need          # the batch splits its KV ranges
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    ref = torch.empty_like(q)
    ref.fill_(0)
    sm.tree_attn(dt, trees, kv, cfg.n_q, q, ref, ws=ws, ws_bytes=need)
    got = torch.empty_like(q)
    got.fill_(0)
    sm.tree_attn_noalloc(dt, trees, kv, cfg.n_q, q, got)
    torch.cuda.synchronize()
    say(f"[noalloc] {cfg.name}: B={cfg.B} sumN={wl.total_nodes} scratch used {need} bytes")
    return runner, ref, got, need


def test_tree_attn_noalloc_matches_workspace_call():
    import torch
    assert torch.cuda.is_available()
    from paper_2506_01986_amd import specmemo as sm
    sm.load()
    # first call: the 70B-shaped batch (GQA 64/8, ragged KV lengths 512..4096)
    big = synth.make(configs.get("llama2_70b_b10"), with_heads=False)
    # second call, smaller: three sequences, one long enough to split, MHA
    cfg = configs.Config(name="noalloc_small", dtype="bf16", B=3, n_q=4, n_kv=4, head_dim=128, hidden=64,
                         vocab=100, n_heads=4, topk=(10, 10, 10, 10), tree="T64", kv_len=(1, 1), seed=5, w_std=0.05)
    rng = np.random.default_rng(5)
    small = synth.make(cfg, trees=[synth.t64(), synth.random_tree(rng, 20), synth.t16()], lens=[6000, 33, 700],
                       with_heads=False)
    sizes = []
    for wl in (big, small):
        runner, ref, got, need = _run_both(torch, wl)
        sizes.append(need)
        # the same kernels and split: the two entry points agree bit for bit
        assert torch.equal(ref.view(torch.int16), got.view(torch.int16)), wl.cfg.name
        # and the result is the oracle's, on every row of the small batch, sampled rows of the big one
        out = synth.storage_to_f64(runner.to_host_storage(got, wl.cfg.dtype), wl.cfg.dtype)
        cfg = wl.cfg
        if wl is big:
            r = np.random.default_rng(0)
            sel = np.stack([r.integers(0, wl.total_nodes, 3000), r.integers(0, cfg.n_q, 3000)], axis=1).astype(np.int32)
            refo = oracle.tree_attn(wl.q, wl.pool_k, wl.pool_v, wl.node_off, wl.parent, wl.lens, wl.seq_base,
                                    cfg.n_kv, sel=sel)
            o = out[sel[:, 0], sel[:, 1]]
        else:
            refo = oracle.tree_attn(wl.q, wl.pool_k, wl.pool_v, wl.node_off, wl.parent, wl.lens, wl.seq_base, cfg.n_kv)
            o = out
        atol, rtol = TOL[cfg.dtype]
        assert np.all(np.abs(o - refo) <= atol + rtol * np.abs(refo)), cfg.name
    assert sizes[1] < sizes[0]
