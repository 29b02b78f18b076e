"""Benchmark of one tree-verification step on one MI355X.

A step is the whole hot path over one batch: Medusa-head projection + top-k +
tree assembly, tree-masked attention, greedy acceptance and in-place KV
compaction, on synthetic inputs already resident in HBM; the timed step makes
three calls (acceptance and compaction fused in one), and the same step
through the four stage calls, and with the attention on a second stream
concurrent with the projection, is timed beside it.  The bf16 head weights
are packed once into the projection's streaming order before timing (a
load-time step: the heads are fixed for a model); every step reads all of them.  Default workload: the
Llama-2-70B-shaped batch of 10 sequences (64 query / 8 KV heads x 128, hidden
8192, vocab 32000, 4 heads, 64-node tree, KV lengths U[512, 4096], slabs capped
at 1.1 x live tokens).

The headline is timed with cold caches: the per-step buffers (queries, KV
pool, base logits, outputs, workspace) have several replicas, step k runs on
replica k mod R, and R replicas exceed twice the 256 MB MALL, so no step finds
its data in the caches; the same step on one replica (warm) is reported
beside it.

Prints one JSON line: the step throughput in verified tree tokens/s (sum of the
tree sizes / step time), per-stage times and achieved bandwidth from HIP events
on the stream the kernels run on, the roofline entry of the dominant kernel
(the head projection, timed by itself over back-to-back launches), and the CPU
oracle's throughput on the same workload; then the padded-batching variant, a
multi-step decode run and the memory-budget plan on the same batch.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "fp32": 157.3}   # MI355X dense matrix bf16 / fp32 vector, published
METRIC = "verified tree tokens/sec per verify step; achieved HBM GB/s vs peak"
# Kernels each stage launches through the C ABI (for matching rocprofv3 traces).
STAGE_KERNELS = {"medusa_topk": ["head_logits_packed", "topk_rows"],
                 "tree_attn": ["tree_attn_bf16", "tree_attn_combine"],
                 "accept": ["row_argbest_all", "accept_walk"], "kv_compact": ["kv_compact_kernel"],
                 "accept_compact": ["row_argbest_all", "accept_walk_compact"]}
FP32_STAGE_KERNELS = {"medusa_topk": ["head_logits_f32", "topk_rows"], "tree_attn": ["tree_attn_f32"]}


def stage_kernels(stage, dtype):
    """The kernels of a stage for this dtype (the fp32 workload has kernels of its own)."""
    return FP32_STAGE_KERNELS.get(stage, STAGE_KERNELS[stage]) if dtype == "fp32" else STAGE_KERNELS[stage]


# Sources whose text decides a stage's kernels (with the shared device.h and
# internal.h): a counter summary is used only while their hash is unchanged.
STAGE_SOURCES = {"medusa_topk": ["medusa_topk.hip"], "tree_attn": ["tree_attn.hip"],
                 "accept": ["accept.hip"], "kv_compact": ["kv_compact.hip", "compact_rows.h"],
                 "accept_compact": ["accept.hip", "compact_rows.h"], "head_logits_packed": ["medusa_topk.hip"]}
# The dominant kernel of a stage, timed by itself for the roofline entry.
DOMINANT_KERNEL = {"medusa_topk": "head_logits_packed"}


def source_sha(stage):
    import hashlib
    h = hashlib.sha256()
    for name in STAGE_SOURCES[stage] + ["device.h", "internal.h"]:
        h.update(open(os.path.join(ROOT, "paper_2506_01986_amd", "csrc", name), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(stage, workload):
    """HBM bytes per launch of a stage from a committed counter summary, or None.

    profiles/<stage>_<workload>_traffic.txt holds "key: value" lines written from
    two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) scaled by the same counters
    on a device copy of known size; it is used only while the stage's kernel
    source still has the recorded hash.
    """
    path = os.path.join(ROOT, "profiles", f"{stage}_{workload}_traffic.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256_16") != source_sha(stage):
        return None
    return int(float(kv["hbm_bytes_per_launch"]))


def algorithmic_bytes(wl, acc):
    """Bytes each stage must move at minimum.

    medusa_topk: the l*w*hidden head weights, the hidden states, the top-k
      lists and the tree tokens.
    tree_attn: each sequence's committed and tree K/V rows once (2 * n_kv *
      head_dim elements per row) plus the queries read and outputs written.
    accept: every node's logit row (sum N_b * vocab * s: a node's row decides
      whether its children are accepted, and which nodes end up on the path
      is known only after reading them) and the node tokens.
    kv_compact: the accepted rows of K and V, read and written once.
    """
    cfg = wl.cfg
    s = cfg.elem_bytes
    sumN = wl.total_nodes
    a = cfg.n_heads * cfg.vocab * cfg.hidden * s + cfg.B * cfg.hidden * s \
        + cfg.B * cfg.n_heads * cfg.kmax * 8 + sumN * 4
    kv_rows = int(np.sum(wl.lens)) + sumN
    b = kv_rows * 2 * cfg.n_kv * cfg.head_dim * s + 2 * sumN * cfg.n_q * cfg.head_dim * s
    c = sumN * cfg.vocab * s + sumN * 4
    d = 2 * int(np.sum(acc + 1)) * 2 * cfg.n_kv * cfg.head_dim * s
    return {"medusa_topk": a, "tree_attn": b, "accept": c, "kv_compact": d}


def projection_kernel(torch, sm, step, cfg, steps):
    """Average duration of the head projection kernel alone (the dominant
    kernel of stage a): `steps` back-to-back launches through
    specmemo_head_logits on the kernels' stream, HIP events at both ends.
    Returns (ms, algorithmic bytes: weights + hidden states read, fp32 logits
    written)."""
    z = torch.empty((cfg.B, cfg.n_heads, cfg.vocab), dtype=torch.float32, device="cuda")

    def call():
        sm.head_logits(step.dt, cfg.B, cfg.hidden, cfg.vocab, cfg.n_heads, step.h, step.head_w, z,
                       head_layout=step.head_layout)
    for _ in range(2):
        call()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        call()
    e1.record()
    torch.cuda.synchronize()
    s = cfg.elem_bytes
    nbytes = cfg.n_heads * cfg.vocab * cfg.hidden * s + cfg.B * cfg.hidden * s + cfg.B * cfg.n_heads * cfg.vocab * 4
    return e0.elapsed_time(e1) / steps, nbytes


def attention_flops(wl):
    """QK^T and PV products of stage (b): 4 d per (query row, visible key); a
    node at depth t sees its L_b committed keys and t + 1 tree rows."""
    cfg = wl.cfg
    keys = 0
    for b in range(cfg.B):
        n0, n1 = int(wl.node_off[b]), int(wl.node_off[b + 1])
        keys += int(np.sum(int(wl.lens[b]) + wl.depth[n0:n1].astype(np.int64) + 1))
    return 4 * cfg.head_dim * cfg.n_q * keys


def cpu_baseline(wl, min_seconds=10.0, max_reps=20, budget=None):
    """The oracle on the same workload, timed on this host's cores.

    The whole step is repeated until at least `min_seconds` of oracle time have
    passed (at most `max_reps` times); the mean is reported.  `budget`
    (device bytes, default tree, model terms) adds the oracle's time for the
    two plans whose library times the budget report gives.
    """
    out = {}
    if budget is not None:
        from oracle import budget as ob
        device_bytes, tree, model = budget
        for name, mem in (("fits", device_bytes), ("exhaustive", 0)):
            t0 = time.perf_counter()
            for _ in range(20):
                ob.plan_budget(mem, batch=wl.cfg.B, default_tree=tuple(map(list, tree)), **model)
            out[name] = round((time.perf_counter() - t0) / 20 * 1e6, 1)
    reps, total, stage_tot = 0, 0.0, np.zeros(4)
    while reps < max_reps and (reps == 0 or total < min_seconds):
        secs, stages = _oracle_step(wl)
        reps += 1
        total += secs
        stage_tot += stages
    import oracle
    cores = oracle.threads()
    mean = total / reps
    # one thread, on the two small workloads (one step each)
    from paper_2506_01986_amd import configs, synth
    single = {}
    oracle.threads(1)
    try:
        for name in ("tiny_fp32", "llama2_7b_b1"):
            w = synth.make(configs.get(name))
            secs, _ = _oracle_step(w)
            single[name] = {"value": round(w.total_nodes / secs, 2), "unit": "tokens/s",
                            "seconds_per_step": round(secs, 4)}
    finally:
        oracle.threads(cores)
    return {"value": wl.total_nodes / mean, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"the whole step on the same workload ({wl.total_nodes} tree tokens, all stages, fp64), "
                      f"{reps} repetitions on {cores} threads; single_thread: one step of the tiny and 7B-shaped "
                      f"workloads on one thread",
            "cpu_model": cpu_model(), "seconds": round(total, 3), "seconds_per_step": round(mean, 3),
            "stage_seconds": {n: round(float(t) / reps, 3)
                              for n, t in zip(["medusa_topk", "tree_attn", "accept", "kv_compact"], stage_tot)},
            "single_thread": single,
            **({"budget_plan_us": out} if out else {})}


def cpu_model():
    """The host CPU's model name (as lscpu reports it, from /proc/cpuinfo)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def _oracle_step(wl):
    import oracle
    cfg = wl.cfg
    t0 = time.perf_counter()
    z = oracle.head_logits(wl.hidden, wl.head_w)
    ids, _ = oracle.heads_topk(z, cfg.topk, cfg.kmax)
    tok = oracle.tree_tokens(wl.node_off, wl.depth, wl.rank, wl.root_tok, ids)
    t1 = time.perf_counter()
    oracle.tree_attn(wl.q, wl.pool_k, wl.pool_v, wl.node_off, wl.parent, wl.lens, wl.seq_base, cfg.n_kv)
    t2 = time.perf_counter()
    from paper_2506_01986_amd import synth
    lg = synth.planted_logits(wl, tok)
    t3 = time.perf_counter()
    acc, path, _ = oracle.accept_greedy(lg, tok, wl.node_off, wl.parent, wl.depth, cfg.n_heads + 1)
    K, V = wl.pool_k.copy(), wl.pool_v.copy()
    t4 = time.perf_counter()
    oracle.kv_compact(K, V, wl.seq_base, wl.lens, acc, path)
    t5 = time.perf_counter()
    stages = np.array([t1 - t0, t2 - t1, t4 - t3, t5 - t4])
    return float(stages.sum()), stages


def padded_report(torch, cfg, wl, step, steps, history=150):
    # at most depth + 1 tokens per step: every sequence keeps a prompt
    history = min(history, int(np.min(wl.lens)) // (cfg.n_heads + 1))
    """The paper's padded batching (Sec. 3.3) on the same batch, for
    comparison with compaction: the same real tokens per sequence after
    `history` padded decode steps (pad tokens interleaved in each cache), one
    step = head projection, attention with the pad mask, acceptance, padded
    update.  Same heads, queries, trees and planted logits as the ragged step."""
    from paper_2506_01986_amd import runner, synth
    rng = np.random.default_rng(cfg.seed + 1000)
    p = cfg.p_accept if cfg.p_accept is not None else float(np.mean(cfg.p_range))
    rows, slab = synth.padded_history(rng, wl.lens, history, p, cfg.n_heads)
    wp = synth.make(cfg, lens=rows, with_heads=False)
    wp.head_w, wp.hidden = wl.head_w, wl.hidden
    flags = synth.pool_key_flags(wp, slab)
    sp = runner.VerifyStep(wp, key_valid=flags)
    sp.base_logits = step.base_logits
    for _ in range(3):
        sp.run_padded()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
    stages = [sp.medusa_topk, sp.tree_attn_padded, sp.accept, sp.kv_pad_update]
    for k in range(steps):
        ev[k][0].record()
        for j, fn in enumerate(stages):
            fn()
            ev[k][j + 1].record()
    torch.cuda.synchronize()
    t = np.array([[ev[k][j].elapsed_time(ev[k][j + 1]) for j in range(4)] for k in range(steps)])
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        sp.run_padded()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    pads = int(np.sum(rows) - np.sum(wl.lens))
    row_bytes = 2 * cfg.n_kv * cfg.head_dim * cfg.elem_bytes          # K and V of one layer
    attn_bytes = (int(np.sum(rows)) + wp.total_nodes) * row_bytes + 2 * wp.total_nodes * cfg.n_q * cfg.head_dim * cfg.elem_bytes
    ta = float(t[:, 1].mean())
    return {"history_steps": history, "kv_rows": int(np.sum(rows)), "pad_rows": pads,
            "pad_frac": round(pads / float(np.sum(rows)), 4),
            "kv_bytes_all_layers": int((np.sum(rows) + wp.total_nodes) * row_bytes * cfg.layers),
            "ms_per_step": round(ms, 5), "value": round(wp.total_nodes / (ms * 1e-3), 1),
            "stages_ms": {n: round(float(t[:, j].mean()), 5) for j, n in
                          enumerate(["medusa_topk", "tree_attn_padded", "accept", "kv_pad_update"])},
            "tree_attn_padded": {"ms": round(ta, 5), "algorithmic_bytes": attn_bytes,
                                 "GBps": round(attn_bytes / (ta * 1e-3) / 1e9, 1)}}


def measured_peaks(torch, reps=10):
    """What this device reaches outside the library, to set the spec peaks in
    context: a 2 GiB device-to-device copy (bytes read + written per second)
    and an 8192^3 bf16 matrix product through torch (the vendor library).
    Neither replaces the spec peaks of the roofline entry."""
    n = 1 << 31
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    src.fill_(1)
    dst = torch.empty_like(src)
    a = torch.randn(8192, 8192, device="cuda", dtype=torch.bfloat16)
    b = torch.randn(8192, 8192, device="cuda", dtype=torch.bfloat16)

    def timed(fn):
        for _ in range(2):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3
    t_copy = timed(lambda: dst.copy_(src))
    t_mm = timed(lambda: torch.matmul(a, b))
    del src, dst, a, b
    return {"copy_GBps": round(2 * n / t_copy / 1e9, 1), "copy_bytes": 2 * n,
            "gemm_bf16_TFLOPs": round(2 * 8192 ** 3 / t_mm / 1e12, 1), "gemm_shape": [8192, 8192, 8192]}


def decode_report(torch, cfg, wl, steps=48, warmup=3):
    """Multi-step decoding on the same batch: residual-block heads, the
    sampled next token, trees sized each step from the slabs' free rows (each
    slab has 64 + U[0, 160) free rows for the run, so some trees shrink), the
    next token chained as the next root, one host read-back per step.  The
    base model's per-step outputs (hidden states, queries, tree K/V rows,
    logits) are Gaussian draws made on the device before timing, and so are
    the planted walks on full-size trees; the host planning, the walks on
    pruned trees and the read-back are inside the timed loop.  The run is
    timed without events, then repeated with an event after every phase for
    the phase table."""
    from paper_2506_01986_amd import runner, synth
    rng = np.random.default_rng(cfg.seed + 2000)
    room = (64 + rng.integers(0, 160, cfg.B)).astype(np.int32)
    nmax = cfg.B * synth.t64().n
    gen = torch.Generator(device="cuda")
    gen.manual_seed(cfg.seed + 2000)
    bf = torch.bfloat16
    rnd = lambda *shape: torch.randn(*shape, generator=gen, device="cuda", dtype=bf)
    pre = [dict(h=rnd(cfg.B, cfg.hidden), q=rnd(nmax, cfg.n_q, cfg.head_dim), k=rnd(cfg.n_kv, nmax, cfg.head_dim),
                v=rnd(cfg.n_kv, nmax, cfg.head_dim), lg=rnd(nmax, cfg.vocab)) for _ in range(warmup + steps)]

    def run(timing):
        # the same run each time: fresh slabs, the same draws
        setup = synth.decode_setup(cfg, cfg.seed + 2000, synth.t64(), room, resblock=True, temperature=0.8,
                                   lens=wl.lens, head_w=wl.head_w)
        loop = runner.DecodeLoop(setup, keep_logits=False, timing=timing)
        prng = np.random.default_rng(cfg.seed + 2001)
        # the planted walks on full-size trees, drawn before timing like the
        # other model outputs; a pruned tree's walk is drawn when it is needed
        full = [synth.plant_walks([setup.default] * cfg.B, setup.p_accept, prng)[0] for _ in range(warmup + steps)]

        def inputs_for(t, plan):
            seqs, sizes = plan
            plans = [full[t][b] if n == setup.default.n else
                     synth.plant_walks([synth.tree_prefix(setup.default, n)], setup.p_accept[[b]], prng)[0][0]
                     for b, n in zip(seqs, sizes)]
            n, x = int(sum(sizes)), pre[t]
            return synth.StepInputs(hidden=x["h"][:len(seqs)], q=x["q"][:n], tree_k=x["k"][:, :n],
                                    tree_v=x["v"][:, :n], base_logits=x["lg"][:n], plans=plans)

        for t in range(warmup):
            plan = loop.plan()
            loop.step(t, inputs_for(t, plan), record=False, plan=plan)
        torch.cuda.synchronize()
        loop.events.clear()
        acc_tokens = tree_tokens = done = 0
        w0 = time.perf_counter()
        for t in range(warmup, warmup + steps):
            plan = loop.plan()
            if not plan[0]:
                break
            rec = loop.step(t, inputs_for(t, plan), record=False, plan=plan)
            acc_tokens += int(np.sum(rec["acc"] + 1))
            tree_tokens += int(sum(rec["sizes"]))
            done += 1
        return time.perf_counter() - w0, done, acc_tokens, tree_tokens, loop, setup

    # the loop's own time, then the same run again with an event after every phase
    wall, done, acc_tokens, tree_tokens, loop, setup = run(False)
    wall_ev, done_ev, *_, loop_ev, _ = run(True)
    phases = loop_ev.phase_ms()
    ph = {k: float(np.mean([e[k] for e in phases])) for k in phases[0]}
    rb_bytes = cfg.n_heads * cfg.hidden * cfg.hidden * cfg.elem_bytes
    return {"steps": done, "ms_per_step": round(wall / done * 1e3, 4),
            "tree_tokens_per_step": round(tree_tokens / done, 1),
            "accepted_tokens_per_step": round(acc_tokens / done, 2),
            "accepted_tokens_per_s": round(acc_tokens / wall, 1),
            "value": round(tree_tokens / wall, 1),
            "full_slabs": int(np.sum(loop.lens >= setup.seq_cap)),
            "ms_per_step_with_phase_events": round(wall_ev / done_ev * 1e3, 4),
            "phase_ms": {k: round(v, 5) for k, v in ph.items()},
            "resblock": {"ms": round(ph["resblock"], 5), "weight_bytes": rb_bytes,
                         "GBps": round(rb_bytes / (ph["resblock"] * 1e-3) / 1e9, 1),
                         "hbm_frac": round(rb_bytes / (ph["resblock"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}}


def budget_model(cfg, wl):
    """The default tree and the model terms of Alg. 1's plan for this workload."""
    tree = (wl.trees[0].parent, wl.trees[0].depth, wl.trees[0].rank)
    model = dict(base_model_bytes=cfg.params * cfg.elem_bytes, head_bytes=cfg.hidden * cfg.vocab * cfg.elem_bytes,
                 layers=cfg.layers, n_kv=cfg.n_kv, head_dim=cfg.head_dim, vocab=cfg.vocab,
                 elem_bytes=cfg.elem_bytes, query_count=1, query_length=int(cfg.kv_len[1]),
                 default_heads=cfg.n_heads)
    return tree, model


def budget_report(cfg, wl, device_bytes, reps=2000):
    """The memory model and Alg. 1's plan for the workload's model on this
    device (host calls of the library), with their host times (the oracle's
    times for the same plans are part of the CPU baseline)."""
    from paper_2506_01986_amd import specmemo as sm
    tree, model = budget_model(cfg, wl)
    plan = sm.plan_budget(device_bytes, batch=cfg.B, default_tree=tree, **model)
    # the largest batch of full-length sequences that keeps the default tree and heads
    lo, hi = 0, 1 << 20
    while lo < hi:
        mid = (lo + hi + 1) // 2
        ok = sm.plan_budget(device_bytes, batch=mid, default_tree=tree, **model)["kind"] == sm.PLAN_DEFAULT
        lo, hi = (mid, hi) if ok else (lo, mid - 1)
    # timing: the plan that fits at once and the one that searches every pruning
    timings = {}
    for name, mem in (("fits", device_bytes), ("exhaustive", 0)):
        t0 = time.perf_counter()
        for _ in range(reps):
            sm.plan_budget(mem, batch=cfg.B, default_tree=tree, **model)
        timings[name] = {"lib_us": round((time.perf_counter() - t0) / reps * 1e6, 2)}
    sizes = sm.plan_tree_sizes(wl.lens, wl.seq_cap, int(wl.trees[0].n))
    t0 = time.perf_counter()
    for _ in range(reps):
        sm.plan_tree_sizes(wl.lens, wl.seq_cap, int(wl.trees[0].n))
    sizes_us = (time.perf_counter() - t0) / reps * 1e6
    per_layer_pool = 2 * wl.cap_total * cfg.n_kv * cfg.head_dim * cfg.elem_bytes
    return {"device_bytes": int(device_bytes), "model_bytes": model["base_model_bytes"],
            "head_bytes": model["head_bytes"], "plan": plan, "max_batch_default_tree": lo,
            "plan_time": timings, "tree_sizes": [int(x) for x in sizes], "tree_sizes_us": round(sizes_us, 2),
            "pool_bytes_all_layers": int(per_layer_pool * cfg.layers),
            "eq1_bytes_live_tokens": sm.mem_kv_bytes(cfg.layers, 1, cfg.n_kv, cfg.head_dim,
                                                     int(np.sum(wl.lens) + wl.total_nodes), cfg.elem_bytes)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--config", default="llama2_70b_b10")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-padded", action="store_true", help="skip the padded-batching comparison")
    ap.add_argument("--no-decode", action="store_true", help="skip the multi-step decode run")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="also run a device-to-device copy of BYTES (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the verify step is a single-GPU path here (asked for --gpus {args.gpus}). "
              "The batch shards by sequence with no exchange; run one process per GPU with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2506_01986_amd import configs, runner, specmemo as sm, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    sm.load()
    # all work on a stream of its own (default priority); the step's attention
    # runs on a second one
    torch.cuda.set_stream(torch.cuda.Stream())
    cfg = configs.get(args.config)
    print(f"[bench] building {cfg.name}", file=sys.stderr, flush=True)
    wl = synth.make(cfg)
    step = runner.VerifyStep(wl)
    step.medusa_topk()                       # the tree tokens plant the synthetic base-model logits
    torch.cuda.synchronize()
    step.set_base_logits(synth.planted_logits(wl, step.node_tok.cpu().numpy()))
    print("[bench] warmup", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step.run_fused()
        step.run()
        step.run_overlapped()
    torch.cuda.synchronize()

    names = ["medusa_topk", "tree_attn", "accept", "kv_compact"]
    # Replicas of every per-step buffer (queries, pool, base logits, outputs,
    # workspace; the head weights are shared and streamed past the caches
    # anyway): steps rotated over them find none of their data in the 256 MB
    # MALL, as in a full model, where the other layers' weights and caches
    # pass through it between two steps of one layer.
    mall = 256 << 20
    nrep = max(3, -(-2 * mall // step.step_bytes()) + 1)
    reps = [step] + [step.replica() for _ in range(nrep - 1)]
    for r in reps[1:]:
        for _ in range(3):
            r.run_fused()
            r.run_overlapped()
    torch.cuda.synchronize()

    def events(n):
        return [torch.cuda.Event(enable_timing=True) for _ in range(n)]

    def loop_ms(fn_of_k):
        """K calls of fn_of_k(k), HIP events on the kernels' stream at the two ends only."""
        e0, e1 = events(2)
        torch.cuda.synchronize()
        e0.record()
        for k in range(args.steps):
            fn_of_k(k)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / args.steps

    def stage_table(rotate):
        """K four-call steps with an event after every stage: [K, 4] ms."""
        ev = [events(5) for _ in range(args.steps)]
        for k in range(args.steps):
            r = reps[k % nrep] if rotate else step
            ev[k][0].record()
            for j, fn in enumerate([r.medusa_topk, r.tree_attn, r.accept, r.kv_compact]):
                fn()
                ev[k][j + 1].record()
        torch.cuda.synchronize()
        return np.array([[ev[k][j].elapsed_time(ev[k][j + 1]) for j in range(4)] for k in range(args.steps)])

    # The same step through the four stage calls (acceptance and compaction
    # separate), rotated over the replicas; timed first, so that the timed
    # step below runs with the clocks in their steady state.
    print("[bench] four-call step", file=sys.stderr, flush=True)
    unfused_ms = loop_ms(lambda k: reps[k % nrep].run())
    print("[bench] warm steps (one replica)", file=sys.stderr, flush=True)
    unfused_warm_ms = loop_ms(lambda k: step.run())
    warm_ms = loop_ms(lambda k: step.run_fused())
    warm_over_ms = loop_ms(lambda k: step.run_overlapped())
    print("[bench] overlapped step (attention on a second stream)", file=sys.stderr, flush=True)
    over_ms = loop_ms(lambda k: reps[k % nrep].run_overlapped())
    # Timed region (the headline): exactly K steps (projection and top-k,
    # attention, acceptance with the compaction fused in: every stage of the
    # path), step k on replica k mod R, HIP events on the kernels' stream at
    # its two ends only (events between stages would add their own packets).
    print("[bench] timing", file=sys.stderr, flush=True)
    w0 = time.perf_counter()
    ms = loop_ms(lambda k: reps[k % nrep].run_fused())
    wall = time.perf_counter() - w0
    # Per-stage breakdown: K four-call steps with an event after every stage,
    # rotated (cold, as the headline) and on one replica (warm).
    print("[bench] stage breakdown", file=sys.stderr, flush=True)
    per_stage = stage_table(True)
    per_stage_warm = stage_table(False)
    # Typical acceptance (App. A.1, Medusa's default): the fused step and the
    # acceptance stage in that mode, rotated like the headline.
    print("[bench] typical acceptance", file=sys.stderr, flush=True)
    for r in reps:
        r.mode = sm.TYPICAL
    typ_ms = loop_ms(lambda k: reps[k % nrep].run_fused())
    typ_stage = stage_table(True)[:, 2]
    for r in reps:
        r.mode = sm.GREEDY
    # The same step captured once in a HIP graph and replayed K times (no
    # per-launch host work; the kernels and their arguments are those above).
    print("[bench] graph replay", file=sys.stderr, flush=True)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step.run_fused()
    graph.replay()
    torch.cuda.synchronize()
    graph_ms = loop_ms(lambda k: graph.replay())
    del graph
    acc = step.accept_len.cpu().numpy()
    byts = algorithmic_bytes(wl, acc)
    st = {}
    for j, n in enumerate(names):
        t, tw = float(per_stage[:, j].mean()), float(per_stage_warm[:, j].mean())
        gbs = byts[n] / (t * 1e-3) / 1e9
        st[n] = {"ms": round(t, 5), "ms_p10": round(float(np.percentile(per_stage[:, j], 10)), 5),
                 "ms_p90": round(float(np.percentile(per_stage[:, j], 90)), 5),
                 "algorithmic_bytes": int(byts[n]), "GBps": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
                 "ms_warm": round(tw, 5), "hbm_frac_warm": round(byts[n] / (tw * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    fl = attention_flops(wl)
    st["tree_attn"]["flops"] = fl
    st["tree_attn"]["TFLOPs"] = round(fl / (st["tree_attn"]["ms"] * 1e-3) / 1e12, 1)
    st["tree_attn"]["mfma_frac"] = round(st["tree_attn"]["TFLOPs"] / MFMA_PEAK_TFLOPS[cfg.dtype], 4)
    st["tree_attn"]["mfma_frac_warm"] = round(fl / (st["tree_attn"]["ms_warm"] * 1e-3) / 1e12
                                              / MFMA_PEAK_TFLOPS[cfg.dtype], 4)
    ab = byts["tree_attn"] + byts["kv_compact"]
    for key, tab in (("tree_attn+kv_compact", per_stage), ("tree_attn+kv_compact_warm", per_stage_warm)):
        at = float((tab[:, 1] + tab[:, 3]).mean())
        st[key] = {"ms": round(at, 5), "GBps": round(ab / (at * 1e-3) / 1e9, 1),
                   "hbm_frac": round(ab / (at * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    tt = float(typ_stage.mean())
    st["accept_typical"] = {"ms": round(tt, 5), "algorithmic_bytes": int(byts["accept"]),
                            "GBps": round(byts["accept"] / (tt * 1e-3) / 1e9, 1),
                            "hbm_frac": round(byts["accept"] / (tt * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    dom = max(names, key=lambda n: st[n]["ms"])
    if DOMINANT_KERNEL.get(dom) == "head_logits_packed" and step.head_layout == sm.HEADS_PACKED:
        print("[bench] projection kernel alone", file=sys.stderr, flush=True)
        kms, kbytes = projection_kernel(torch, sm, step, cfg, args.steps)
        kgbs = kbytes / (kms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "kernel": "head_logits_packed", "stage": dom, "achieved": round(kgbs, 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(kgbs / HBM_PEAK_GBS, 4),
                    "traffic": measured_traffic("head_logits_packed", cfg.name), "algorithmic_bytes": kbytes,
                    "ms": round(kms, 5), "source_sha256_16": source_sha("head_logits_packed")}
    elif dom == "tree_attn" and cfg.dtype == "bf16":
        # attention above the ridge point (FLOP per algorithmic byte > 2.5 PFLOP/s / 8 TB/s): matrix-core bound
        roofline = {"bound": "mfma", "kernel": dom, "kernels": stage_kernels(dom, cfg.dtype), "achieved": st[dom]["TFLOPs"],
                    "peak": MFMA_PEAK_TFLOPS[cfg.dtype], "unit": "TFLOP/s", "frac": st[dom]["mfma_frac"],
                    "traffic": measured_traffic(dom, cfg.name), "algorithmic_flops": st[dom]["flops"],
                    "algorithmic_bytes": st[dom]["algorithmic_bytes"], "ms": st[dom]["ms"],
                    "source_sha256_16": source_sha(dom)}
    else:
        roofline = {"bound": "hbm", "kernel": dom, "kernels": stage_kernels(dom, cfg.dtype), "achieved": st[dom]["GBps"],
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": st[dom]["hbm_frac"],
                    "traffic": measured_traffic(dom, cfg.name), "algorithmic_bytes": st[dom]["algorithmic_bytes"],
                    "ms": st[dom]["ms"], "source_sha256_16": source_sha(dom)}
    if args.copy_calibration:
        src = torch.empty(args.copy_calibration, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
    result = {
        "metric": METRIC, "value": round(wl.total_nodes / (ms * 1e-3), 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype,
        "data": "synthetic (seeded Gaussian weights/activations/KV, planted acceptance)",
        "config": {"workload": f"{cfg.name}: B={cfg.B}, {cfg.n_q}q/{cfg.n_kv}kv x {cfg.head_dim}, hidden {cfg.hidden}, "
                               f"vocab {cfg.vocab}, {cfg.n_heads} heads top-{cfg.kmax}, tree {cfg.tree}, "
                               f"KV {cfg.kv_len_dist} {list(cfg.kv_len)}, pool {cfg.pool}",
                   "batch": cfg.B, "tree_tokens": wl.total_nodes, "kv_tokens": int(np.sum(wl.lens)),
                   "accepted_tokens": int(np.sum(acc + 1))},
        "roofline": roofline,
        "accepted_tokens_per_s": round(float(np.sum(acc + 1)) / (ms * 1e-3), 1),
        "wall_ms_per_step": round(wall / args.steps * 1e3, 5),
        "caches": {"headline": f"cold: step k runs on replica k mod {nrep} of the per-step buffers "
                               f"({step.step_bytes()} bytes each; the MALL holds 256 MB)",
                   "replicas": nrep, "replica_bytes": step.step_bytes()},
        "warm": {"ms_per_step": round(warm_ms, 5), "value": round(wl.total_nodes / (warm_ms * 1e-3), 1),
                 "note": "the same step, every step on one replica (its pool stays in the MALL)"},
        "overlapped_step": {"ms_per_step": round(over_ms, 5), "ms_per_step_warm": round(warm_over_ms, 5),
                            "note": "the attention on a second stream, concurrent with the projection and top-k "
                                    "(they share no data in this synthetic step; in a full model the queries "
                                    "come from the tree tokens), rotated like the headline; the two kernels "
                                    "then share the compute units and the projection's stream slows by about "
                                    "the attention's time"},
        "typical": {"ms_per_step": round(typ_ms, 5), "value": round(wl.total_nodes / (typ_ms * 1e-3), 1),
                    "accept_stage_ms": st["accept_typical"]["ms"], "temperature": step.temperature,
                    "eps": step.eps, "delta": step.delta},
        "ms_per_step_with_stage_events": round(float(per_stage.sum(axis=1).mean()), 5),
        "graph": {"ms_per_step": round(graph_ms, 5), "value": round(wl.total_nodes / (graph_ms * 1e-3), 1),
                  "note": "one replica (warm)"},
        "step_calls": ["specmemo_medusa_topk", "specmemo_tree_attn", "specmemo_accept_compact"],
        "four_call_step": {"calls": ["specmemo_medusa_topk", "specmemo_tree_attn", "specmemo_accept",
                                     "specmemo_kv_compact"],
                           "ms_per_step": round(unfused_ms, 5), "value": round(wl.total_nodes / (unfused_ms * 1e-3), 1),
                           "ms_per_step_warm": round(unfused_warm_ms, 5)},
        "stages": st,
    }
    if not args.copy_calibration:       # a counter run keeps the calibration copy the only large copy
        print("[bench] measured peaks (copy, library GEMM)", file=sys.stderr, flush=True)
        mp = measured_peaks(torch)
        if roofline["unit"] == "GB/s":
            mp["dominant_kernel_frac_of_copy"] = round(roofline["achieved"] / mp["copy_GBps"], 4)
        if cfg.dtype == "bf16":
            mp["attention_frac_of_gemm"] = round(st["tree_attn"]["TFLOPs"] / mp["gemm_bf16_TFLOPs"], 4)
        result["measured_peaks"] = mp
    if not args.no_padded:
        print("[bench] padded batching variant", file=sys.stderr, flush=True)
        pr = padded_report(torch, cfg, wl, step, args.steps)
        pr["kv_bytes_all_layers_compacted"] = int((np.sum(wl.lens) + wl.total_nodes) * 2 * cfg.n_kv * cfg.head_dim
                                                  * cfg.elem_bytes * cfg.layers)
        pr["step_time_vs_compaction"] = round(pr["ms_per_step"] / unfused_warm_ms, 4)   # both four-call, warm
        result["padded"] = pr
    if not args.no_decode and cfg.dtype == "bf16":
        print("[bench] multi-step decode", file=sys.stderr, flush=True)
        result["decode"] = decode_report(torch, cfg, wl)
    if cfg.params:
        print("[bench] memory budget plan (host)", file=sys.stderr, flush=True)
        result["budget"] = budget_report(cfg, wl, torch.cuda.get_device_properties(0).total_memory)
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        budget = None
        if cfg.params:
            budget = (torch.cuda.get_device_properties(0).total_memory, *budget_model(cfg, wl))
        result["cpu_baseline"] = cpu_baseline(wl, budget=budget)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
