"""Child process of test_attention_tuning_overrides: tree attention on one
GQA batch with long and short sequences (so that the KV range is split; with
the argument "many", 40 of them: more than one launch's arguments hold),
under the tuning variables of the environment it is started with, checked
against the oracle on sampled rows.  Exit status 0 when within tolerance."""

import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import oracle  # noqa: E402
from paper_2506_01986_amd import configs, runner, synth  # noqa: E402


def main():
    import torch
    assert torch.cuda.is_available()
    many = len(sys.argv) > 1 and sys.argv[1] == "many"   # more sequences than one launch's arguments hold
    rng = np.random.default_rng(3)
    if many:
        B = 40
        trees = [synth.random_tree(rng, int(rng.integers(1, 70))) for _ in range(B)]
        lens = [int(x) for x in rng.integers(0, 900, B)]
        lens[3], lens[17], lens[38] = 6000, 4100, 2500
    else:
        B = 4
        trees = [synth.t64(), synth.random_tree(rng, 100), synth.t16(), synth.chain_tree(5)]
        lens = [5000, 1200, 0, 3100]
    cfg = configs.Config(name="override", dtype="bf16", B=B, n_q=16, n_kv=2, head_dim=128, hidden=64, vocab=300,
                         n_heads=4, topk=(10, 10, 10, 10), tree="T64", kv_len=(1, 1), seed=3, w_std=0.05)
    wl = synth.make(cfg, with_heads=False, trees=trees, lens=lens)
    step = runner.VerifyStep(wl)
    step.tree_attn()
    torch.cuda.synchronize()
    out = synth.storage_to_f64(runner.to_host_storage(step.out, "bf16"), "bf16")
    sel = np.array(sorted({(int(rng.integers(wl.total_nodes)), int(rng.integers(cfg.n_q))) for _ in range(300)}
                          | {(int(wl.node_off[b]), 0) for b in range(cfg.B)}), dtype=np.int32)
    ref = oracle.tree_attn(wl.q, wl.pool_k, wl.pool_v, wl.node_off, wl.parent, wl.lens, wl.seq_base, cfg.n_kv, sel=sel)
    got = out[sel[:, 0], sel[:, 1]]
    err = float((np.abs(got - ref) - (1e-2 + 2e-2 * np.abs(ref))).max())
    env = {k: v for k, v in os.environ.items() if k.startswith("SPECMEMO_ATTN")}
    print(f"override {env} B={B}: rows {len(sel)} margin {err:.3g}", flush=True)
    return 0 if err <= 0 else 1


if __name__ == "__main__":
    sys.exit(main())
