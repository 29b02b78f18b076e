"""GPU parity of the decode-loop pieces and of a multi-step decode against the
oracle: residual-block heads, per-head projection inputs, the sampled next
token, and a loop in which trees shrink as slabs fill up and the next token
becomes the next root.  Tolerances as for the single step; token ids,
lengths, paths and the final cache bit-exact (sampled tokens: except where two
Gumbel keys lie within fp32 rounding of each other)."""

import numpy as np
import pytest

import oracle
from oracle import budget as ob
from oracle import decode as odec
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


def near_tie(best, second):
    return abs(float(best) - float(second)) <= 1e-5 * (1.0 + abs(float(best)))


@pytest.mark.parametrize("dtype,B,hidden", [("bf16", 10, 2048), ("bf16", 17, 512), ("fp32", 3, 96)])
def test_resblock_and_per_head_projection(torch_cuda, dtype, B, hidden):
    torch = torch_cuda
    from paper_2506_01986_amd import runner, specmemo as sm
    rng = np.random.default_rng(hidden + B)
    n_heads, vocab = 4, 1000
    st = lambda n, s: synth._store((s * rng.standard_normal(n)).astype(np.float32), dtype)
    h = st(B * hidden, 1.0).reshape(B, hidden)
    w1 = st(n_heads * hidden * hidden, 0.02).reshape(n_heads, hidden, hidden)
    b1 = st(n_heads * hidden, 0.02).reshape(n_heads, hidden)
    W = st(n_heads * vocab * hidden, 0.05).reshape(n_heads, vocab, hidden)
    say(f"[decode] resblock {dtype} B={B} hidden={hidden}")
    dt = sm.BF16 if dtype == "bf16" else sm.FP32
    hd, w1d, b1d, Wd = (runner.to_device(x, dtype, "cuda") for x in (h, w1, b1, W))
    layout = sm.HEADS_ROWMAJOR
    if dt == sm.BF16:
        pk = torch.empty(sm.packed_heads_bytes(dt, n_heads, hidden, hidden), dtype=torch.uint8, device="cuda")
        sm.pack_heads(dt, n_heads, hidden, hidden, w1d, pk)
        w1d, layout = pk, sm.HEADS_PACKED
    out = torch.empty((n_heads, B, hidden), dtype=hd.dtype, device="cuda")
    sm.medusa_resblock(dt, B, hidden, n_heads, hd, w1d, b1d, out, w1_layout=layout)
    torch.cuda.synchronize()
    got = synth.storage_to_f64(runner.to_host_storage(out, dtype), dtype)
    ref64 = oracle.resblock(h, w1, b1)
    assert close(got, ref64, dtype) <= 0
    # the projection reading each head's own input
    hh = oracle.to_storage(ref64, dtype)
    z64 = np.concatenate([oracle.head_logits(hh[i], W[i:i + 1]) for i in range(n_heads)], axis=1)
    node_off = np.arange(B + 1, dtype=np.int32)             # single-node trees
    zeros = np.zeros(B, np.int32)
    tr = sm.Trees(node_off, np.full(B, -1, np.int32), zeros, zeros, device="cuda")
    hin = runner.to_device(hh, dtype, "cuda")
    z = torch.empty((B, n_heads, vocab), dtype=torch.float32, device="cuda")
    ids = torch.empty((B, n_heads, 4), dtype=torch.int32, device="cuda")
    tok = torch.empty(B, dtype=torch.int32, device="cuda")
    root = torch.zeros(B, dtype=torch.int32, device="cuda")
    hl = runner.to_device(W, dtype, "cuda")
    wl_layout = sm.HEADS_ROWMAJOR
    if dt == sm.BF16:
        pk2 = torch.empty(sm.packed_heads_bytes(dt, n_heads, vocab, hidden), dtype=torch.uint8, device="cuda")
        sm.pack_heads(dt, n_heads, vocab, hidden, hl, pk2)
        hl, wl_layout = pk2, sm.HEADS_PACKED
    sm.medusa_topk(dt, tr, hidden, vocab, n_heads, (4,) * n_heads, hin, hl, root, ids, tok, logits_out=z,
                   head_layout=wl_layout | sm.HEADS_INPUT_PER_HEAD)
    torch.cuda.synchronize()
    assert close(z.cpu().numpy(), z64, dtype) <= 0


@pytest.mark.parametrize("temperature", [0.3, 1.0, 4.0])
def test_sampled_next_token(torch_cuda, temperature):
    torch = torch_cuda
    from paper_2506_01986_amd import runner, specmemo as sm
    rng = np.random.default_rng(int(temperature * 10))
    B, vocab, n = 40, 32000, 5
    lg = synth._store(rng.standard_normal(B * n * vocab).astype(np.float32), "bf16").reshape(B * n, vocab)
    node_off = np.arange(0, B * n + 1, n, dtype=np.int32)
    chain = synth.chain_tree(n)
    tr = sm.Trees(node_off, np.tile(chain.parent, B), np.tile(chain.depth, B), np.tile(chain.rank, B), device="cuda")
    acc = rng.integers(0, n, B).astype(np.int32)
    path = np.tile(np.arange(n, dtype=np.int32), (B, 1))
    seed, offset = 12345, 67
    ref, best, second = oracle.sample_next(lg, node_off, acc, path, temperature, seed, offset)
    d = lambda x: torch.from_numpy(x).to("cuda")
    nxt = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    lg_d = runner.to_device(lg, "bf16", "cuda")
    sm.sample_next(sm.BF16, tr, vocab, temperature, seed, offset, lg_d, d(acc), d(path), n, nxt)
    # the segmented form (a workspace word per 1024-token segment) draws the same tokens
    wsb = sm.workspace_bytes(sm.WS_SAMPLE, sm.BF16, tr, None, 0, vocab)
    ws = torch.full((wsb,), 0xA5, dtype=torch.uint8, device="cuda")
    nxt_seg = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    sm.sample_next(sm.BF16, tr, vocab, temperature, seed, offset, lg_d, d(acc), d(path), n, nxt_seg, ws=ws,
                   ws_bytes=wsb)
    torch.cuda.synchronize()
    got = nxt.cpu().numpy()
    assert np.array_equal(nxt_seg.cpu().numpy(), got)
    diff = np.nonzero(got != ref)[0]
    say(f"[decode] sampled T={temperature}: {B - len(diff)}/{B} equal, near ties {[int(b) for b in diff]}")
    for b in diff:
        assert near_tie(best[b], second[b]), (b, got[b], ref[b], best[b], second[b])
    assert len(diff) <= 1
    assert len(set(got.tolist())) > B // 2                  # draws, not one repeated argmax


DECODE = {
    # residual-block heads, sampled next token, one slab filling up, one shrinking its trees
    "resblock_sampled": (dict(dtype="bf16", B=3, n_q=8, n_kv=2, hidden=64, vocab=500), [300, 70, 9], True, 0.8, 14),
    # plain heads, greedy next token, GQA with 128-node default tree
    "greedy_t128": (dict(dtype="bf16", B=4, n_q=4, n_kv=1, hidden=48, vocab=700), [400, 140, 30, 400], False, None,
                    10),
    # fp32 path
    "fp32": (dict(dtype="fp32", B=2, n_q=4, n_kv=2, head_dim=64, hidden=40, vocab=333, w_std=1.0), [90, 12], True,
             1.5, 8),
    # typical acceptance (App. A.1) with the sampled next token
    "typical": (dict(dtype="bf16", B=3, n_q=8, n_kv=2, hidden=64, vocab=500), [300, 70, 9], True, 0.8, 10,
                (0.7, 0.09, 0.3)),
    # typical acceptance with vanishing thresholds: every step accepts a deepest node
    "typical_deepest": (dict(dtype="bf16", B=3, n_q=8, n_kv=2, hidden=64, vocab=500), [300, 200, 60], False, None, 8,
                        (0.7, 1e-30, 1e-30)),
}


@pytest.mark.parametrize("name", list(DECODE))
def test_decode_loop(torch_cuda, name):
    from paper_2506_01986_amd import runner
    kw, room, resblock, temperature, steps, *rest = DECODE[name]
    typical = rest[0] if rest else None
    base = dict(name=name, head_dim=128, n_heads=4, topk=(10, 10, 10, 10), tree="T64", kv_len=(5, 200),
                kv_len_dist="uniform", seed=11, w_std=0.05, p_accept=0.7)
    base.update(kw)
    cfg = configs.Config(**base)
    default = synth.t64()
    if name == "greedy_t128":
        default = synth.Tree(*(np.asarray(a, np.int32) for a in ob.build_tree(128, 45, 4, 10)))
    st = synth.decode_setup(cfg, 11, default, room, resblock=resblock, temperature=temperature, typical=typical)
    say(f"[decode] {name}: lens {st.lens.tolist()} caps {st.seq_cap.tolist()} steps {steps}")
    recs, K, V, lens = odec.run(st, steps)
    loop = runner.DecodeLoop(st)
    for rec in recs:
        if name == "greedy_t128":
            # the caller's form (as the benchmark drives it): plan and inputs passed in
            plan = loop.plan()
            trees = [synth.tree_prefix(st.default, n) for n in plan[1]]
            g = loop.step(rec["step"], inputs=synth.decode_step_inputs(st, rec["step"], plan[0], trees), plan=plan)
        else:
            g = loop.step(rec["step"])
        assert g is not None
        assert g["seqs"] == rec["seqs"] and g["sizes"] == rec["sizes"], rec["step"]
        assert close(g["z"], rec["z"], cfg.dtype) <= 0
        assert np.array_equal(g["ids"], rec["ids"]), rec["step"]
        assert np.array_equal(g["tok"], rec["tok"]), rec["step"]
        attn = synth.storage_to_f64(runner.to_host_storage(g["attn"], cfg.dtype), cfg.dtype)
        assert close(attn, rec["attn"], cfg.dtype) <= 0
        assert np.array_equal(g["acc"], rec["acc"]) and np.array_equal(g["path"], rec["path"])
        if temperature is not None:
            # two Gumbel keys within rounding: either draw is correct, and the
            # runs part ways from here
            diff = np.nonzero(g["next_tok"] != rec["next_tok"])[0]
            if len(diff):
                assert all(near_tie(rec["best_key"][i], rec["second_key"][i]) for i in diff), rec["step"]
                say(f"[decode]   step {rec['step']}: sampled near tie, comparison ends")
                return
        assert np.array_equal(g["next_tok"], rec["next_tok"]), rec["step"]
        assert np.array_equal(g["lens"], rec["lens"])
        say(f"[decode]   step {rec['step']}: seqs {rec['seqs']} sizes {rec['sizes']} accepted {(rec['acc'] + 1).tolist()}")
    assert loop.step(len(recs)) is None or len(recs) == steps
    Kg = runner.to_host_storage(loop.k, cfg.dtype)
    Vg = runner.to_host_storage(loop.v, cfg.dtype)
    for b in range(cfg.B):
        s0 = int(st.seq_base[b])
        rows = slice(s0, s0 + int(lens[b]))
        assert np.array_equal(Kg[:, rows].view(np.uint8), K[:, rows].view(np.uint8)), b
        assert np.array_equal(Vg[:, rows].view(np.uint8), V[:, rows].view(np.uint8)), b
