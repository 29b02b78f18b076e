"""Seeded synthetic inputs for the verify step.

This module only draws numbers and lays them out.  It holds none of the
method's arithmetic (no projection, top-k, attention, acceptance or
compaction), so that the CPU oracle and the HIP path can both be fed from it
without sharing any computation.

Stand-ins (the paper's models, Medusa heads and MT-Bench/story prompts are not
available):
  * last hidden state, head weights, queries, K/V rows, base-model logits:
    Gaussian draws (fp32 draws, rounded to bf16 with round-to-nearest-even),
  * committed KV lengths: fixed, uniform or log-uniform per sequence, standing
    in for multi-turn chat history of n queries x m tokens (SpecMemo Eq. 1),
  * candidate trees: the builder's 16- and 64-node trees, or random trees of
    depth <= 4 and arity <= 10 (the 64-node tree reproduces the Medusa row of
    SpecMemo Table 1),
  * base-model acceptance: a planted walk.  From the root, with probability p
    one uniformly chosen child's token is made the argmax (+16) of the parent's
    logit row and the walk continues there; otherwise every child token of the
    current node gets -16 and the walk stops.  The planted walk is therefore the
    accepted path under greedy acceptance.

Random streams: ``SeedSequence(seed).spawn(12)`` in the fixed order of
``STREAMS``; large arrays are drawn in fixed-size chunks, each from its own
spawned child, so the bytes do not depend on the number of threads.
"""

from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Dict, List, Sequence, Tuple

import numpy as np

from .configs import Config

STREAMS = ("lens", "trees", "hidden", "head_w", "root", "q", "k_comm", "v_comm",
           "k_tree", "v_tree", "base_logits", "plant")

CHUNK = 1 << 22          # values per independently seeded chunk
PLANT_HI = 16.0          # exact in bf16 and far above any N(0,1) draw
PLANT_LO = -16.0

# Bit patterns of rows that no kernel may read or write: a quiet NaN with a
# payload for the canary rows between slabs, another for unused slab capacity.
CANARY_BF16 = 0x7FC1
FREE_BF16 = 0x7FA5
CANARY_FP32 = 0x7FC00001
FREE_FP32 = 0x7FA5A5A5


# ----------------------------------------------------------------------------
# Trees (BFS order: parent[n] < n, depth non-decreasing, siblings by rank)
# ----------------------------------------------------------------------------

@dataclass
class Tree:
    parent: np.ndarray   # int32 [N], parent[0] = -1
    depth: np.ndarray    # int32 [N]
    rank: np.ndarray     # int32 [N], index into head depth-1's top-k list

    @property
    def n(self) -> int:
        return int(self.parent.shape[0])


def tree_from_rank_paths(paths: Sequence[Tuple[int, ...]]) -> Tree:
    """Build a BFS-ordered tree from a prefix-closed set of rank paths.

    The root is the empty path.  Within a depth, nodes are ordered by their
    parent's id and then by rank.
    """
    pset = set(tuple(p) for p in paths)
    pset.add(())
    for p in pset:
        for i in range(len(p)):
            if p[:i] not in pset:
                raise ValueError(f"rank path {p} has no parent {p[:i]}")
    ids: Dict[Tuple[int, ...], int] = {(): 0}
    order: List[Tuple[int, ...]] = [()]
    maxd = max(len(p) for p in pset)
    for d in range(1, maxd + 1):
        level = [p for p in pset if len(p) == d]
        level.sort(key=lambda p: (ids[p[:-1]], p[-1]))
        for p in level:
            ids[p] = len(order)
            order.append(p)
    parent = np.array([-1] + [ids[p[:-1]] for p in order[1:]], dtype=np.int32)
    depth = np.array([len(p) for p in order], dtype=np.int32)
    rank = np.array([0] + [p[-1] for p in order[1:]], dtype=np.int32)
    return Tree(parent, depth, rank)


def t16() -> Tree:
    """16-node tree for 3 heads with top-k (4, 2, 2); level sizes 1-4-6-5."""
    parent = [-1, 0, 0, 0, 0, 1, 1, 2, 2, 3, 4, 5, 5, 6, 7, 9]
    rank = [0, 0, 1, 2, 3, 0, 1, 0, 1, 0, 0, 0, 1, 0, 0, 0]
    depth = [0, 1, 1, 1, 1, 2, 2, 2, 2, 2, 2, 3, 3, 3, 3, 3]
    return Tree(np.array(parent, np.int32), np.array(depth, np.int32), np.array(rank, np.int32))


def t64() -> Tree:
    """64-node, 42-leaf tree for 4 heads with top-10; level sizes 1-10-23-23-7.

    Its depth-truncated (leaves / nodes) profile is 10/11, 25/34, 39/57, 42/64,
    the Medusa row of SpecMemo Table 1, and it is the "(64 nodes, 42 sequences)"
    default tree of Alg. 1.  Child counts are listed per rank path.
    """
    kids = {(): 10}
    for r, c in enumerate([6, 5, 3, 3, 2, 2, 1, 1, 0, 0]):
        kids[(r,)] = c
    kids.update({(0, 0): 6, (0, 1): 4, (1, 0): 4, (0, 2): 2, (1, 1): 2, (2, 0): 2,
                 (0, 3): 1, (3, 0): 1, (4, 0): 1})
    kids.update({(0, 0, 0): 3, (0, 0, 1): 2, (0, 1, 0): 1, (1, 0, 0): 1})
    paths = [()]
    for p, c in kids.items():
        paths += [p + (r,) for r in range(c)]
    return tree_from_rank_paths(paths)


def random_tree(rng: np.random.Generator, n: int, max_depth: int = 4, max_kids: int = 10) -> Tree:
    """Random tree of n nodes: each new node picks a uniformly random existing
    node of depth < max_depth with fewer than max_kids children as its parent,
    taking that parent's next free rank; then renumbered to BFS order."""
    paths: List[Tuple[int, ...]] = [()]
    nkids = [0]
    for _ in range(1, n):
        cand = [i for i, p in enumerate(paths) if len(p) < max_depth and nkids[i] < max_kids]
        j = cand[int(rng.integers(len(cand)))]
        paths.append(paths[j] + (nkids[j],))
        nkids[j] += 1
        nkids.append(0)
    return tree_from_rank_paths(paths)


def chain_tree(n: int) -> Tree:
    """Single branch: node i's parent is i-1 (rank 0 at every depth)."""
    return tree_from_rank_paths([tuple([0] * i) for i in range(n)])


def star_tree(n: int) -> Tree:
    """Root plus n-1 children at depth 1."""
    return tree_from_rank_paths([()] + [(r,) for r in range(n - 1)])


def children(t: Tree, u: int) -> List[int]:
    return [c for c in range(t.n) if t.parent[c] == u]


# ----------------------------------------------------------------------------
# Value draws
# ----------------------------------------------------------------------------

_NTHREADS = max(1, min(16, os.cpu_count() or 1))


def normals(ss: np.random.SeedSequence, n: int, std: float = 1.0) -> np.ndarray:
    """n standard-normal fp32 draws times std, chunked over spawned children."""
    nchunk = max(1, (n + CHUNK - 1) // CHUNK)
    kids = ss.spawn(nchunk)
    out = np.empty(n, dtype=np.float32)

    def fill(i):
        lo, hi = i * CHUNK, min(n, (i + 1) * CHUNK)
        g = np.random.Generator(np.random.PCG64(kids[i]))
        g.standard_normal(hi - lo, dtype=np.float32, out=out[lo:hi])
        if std != 1.0:
            out[lo:hi] *= np.float32(std)

    if nchunk == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(_NTHREADS) as ex:
            list(ex.map(fill, range(nchunk)))
    return out


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    return x.astype(np.float32) if dtype == "fp32" else to_bf16_bits(x)


# ----------------------------------------------------------------------------
# Workload
# ----------------------------------------------------------------------------

@dataclass
class Workload:
    cfg: Config
    seed: int
    lens: np.ndarray            # int32 [B] committed KV rows per sequence (L_b)
    trees: List[Tree]
    node_off: np.ndarray        # int32 [B+1]
    parent: np.ndarray          # int32 [sumN], local ids
    depth: np.ndarray           # int32 [sumN]
    rank: np.ndarray            # int32 [sumN]
    hidden: np.ndarray          # [B, hidden]   (float32 or uint16 bf16 bits)
    head_w: np.ndarray | None   # [n_heads, vocab, hidden]
    root_tok: np.ndarray        # int32 [B]
    q: np.ndarray               # [sumN, n_q, d]
    pool_k: np.ndarray          # [n_kv, cap_total, d]
    pool_v: np.ndarray
    seq_base: np.ndarray        # int64 [B] first pool row of each slab
    seq_cap: np.ndarray         # int32 [B] slab capacity in rows
    base_logits: np.ndarray     # [sumN, vocab], before planting
    p_accept: np.ndarray        # float64 [B]
    plan: List[List[Tuple[int, int, float]]]   # per sequence: (u, child, value) local ids
    plan_path: List[List[int]]                 # per sequence: planted walk, local ids
    store_dtype: str = "bf16"

    @property
    def total_nodes(self) -> int:
        return int(self.node_off[-1])

    @property
    def cap_total(self) -> int:
        return int(self.pool_k.shape[1])

    @property
    def max_nodes(self) -> int:
        return int(np.max(np.diff(self.node_off)))

    @property
    def max_depth(self) -> int:
        return int(self.depth.max())

    def tree_of(self, b: int) -> Tree:
        return self.trees[b]


def _lens(cfg: Config, rng: np.random.Generator) -> np.ndarray:
    lo, hi = cfg.kv_len
    if cfg.kv_len_dist == "fixed":
        v = np.full(cfg.B, lo, dtype=np.int64)
    elif cfg.kv_len_dist == "uniform":
        v = rng.integers(lo, hi + 1, size=cfg.B)
    elif cfg.kv_len_dist == "loguniform":
        u = rng.random(cfg.B)
        v = np.rint(np.exp(math.log(lo) + u * (math.log(hi) - math.log(lo)))).astype(np.int64)
        v = np.clip(v, lo, hi)
    else:
        raise ValueError(cfg.kv_len_dist)
    return v.astype(np.int32)


def _trees(cfg: Config, rng: np.random.Generator) -> List[Tree]:
    if cfg.tree == "T16":
        return [t16() for _ in range(cfg.B)]
    if cfg.tree == "T64":
        return [t64() for _ in range(cfg.B)]
    if cfg.tree == "random":
        sizes = [int(cfg.tree_sizes[int(rng.integers(len(cfg.tree_sizes)))]) for _ in range(cfg.B)]
        return [random_tree(rng, n, max_depth=cfg.n_heads, max_kids=min(cfg.topk)) for n in sizes]
    raise ValueError(cfg.tree)


def _caps(cfg: Config, lens: np.ndarray, sizes: np.ndarray) -> np.ndarray:
    if cfg.pool == "exact":
        return (lens + sizes).astype(np.int32)
    if cfg.pool == "cap1.1":
        live = lens.astype(np.int64) + sizes
        return (live + live // 10).astype(np.int32)
    if cfg.pool == "fixed1.1":
        live = lens.astype(np.int64) + max(cfg.tree_sizes)
        return (live + live // 10).astype(np.int32)
    raise ValueError(cfg.pool)


def plant_walks(trees: List[Tree], p: np.ndarray, rng: np.random.Generator):
    plans, paths = [], []
    for b, t in enumerate(trees):
        u, plan, path = 0, [], [0]
        while True:
            kids = children(t, u)
            if not kids:
                break
            if rng.random() < p[b]:
                c = kids[int(rng.integers(len(kids)))]
                plan.append((u, c, PLANT_HI))
                path.append(c)
                u = c
            else:
                plan += [(u, c, PLANT_LO) for c in kids]
                break
        plans.append(plan)
        paths.append(path)
    return plans, paths


def make(cfg: Config, seed: int | None = None, with_heads: bool = True,
         trees: List[Tree] | None = None, lens: Sequence[int] | None = None,
         caps: Sequence[int] | None = None) -> Workload:
    """Build the workload of ``cfg`` from ``seed`` (default: the config's).

    ``trees`` / ``lens`` / ``caps`` (slab rows) override the drawn or derived
    ones (used by special-case tests); ``with_heads=False`` skips the head
    weights.
    """
    seed = cfg.seed if seed is None else seed
    ss = dict(zip(STREAMS, np.random.SeedSequence(seed).spawn(len(STREAMS))))
    rng = {k: np.random.Generator(np.random.PCG64(v)) for k, v in ss.items()}
    B, d, dt = cfg.B, cfg.head_dim, cfg.dtype

    L = _lens(cfg, rng["lens"]) if lens is None else np.asarray(lens, np.int32)
    T = _trees(cfg, rng["trees"]) if trees is None else list(trees)
    assert len(L) == B and len(T) == B
    sizes = np.array([t.n for t in T], dtype=np.int64)
    node_off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    parent = np.concatenate([t.parent for t in T]).astype(np.int32)
    depth = np.concatenate([t.depth for t in T]).astype(np.int32)
    rank = np.concatenate([t.rank for t in T]).astype(np.int32)
    sumN = int(node_off[-1])

    hidden = _store(normals(ss["hidden"], B * cfg.hidden), dt).reshape(B, cfg.hidden)
    head_w = None
    if with_heads:
        head_w = _store(normals(ss["head_w"], cfg.n_heads * cfg.vocab * cfg.hidden, cfg.w_std), dt)
        head_w = head_w.reshape(cfg.n_heads, cfg.vocab, cfg.hidden)
    root_tok = rng["root"].integers(0, cfg.vocab, size=B).astype(np.int32)
    q = _store(normals(ss["q"], sumN * cfg.n_q * d), dt).reshape(sumN, cfg.n_q, d)

    caps = _caps(cfg, L, sizes) if caps is None else np.asarray(caps, np.int32)
    assert np.all(caps.astype(np.int64) >= L.astype(np.int64) + sizes), "a slab must hold its tree"
    base = np.zeros(B, dtype=np.int64)
    row = 1                                   # canary row 0
    for b in range(B):
        base[b] = row
        row += int(caps[b]) + 1               # slab, then a canary row
    cap_total = row
    if dt == "fp32":
        pk = np.full((cfg.n_kv, cap_total, d), CANARY_FP32, dtype=np.uint32)
        free = FREE_FP32
    else:
        pk = np.full((cfg.n_kv, cap_total, d), CANARY_BF16, dtype=np.uint16)
        free = FREE_BF16
    pv = pk.copy()
    kc, vc = ss["k_comm"].spawn(B), ss["v_comm"].spawn(B)
    kt, vt = ss["k_tree"].spawn(B), ss["v_tree"].spawn(B)
    for b in range(B):
        s0, Lb, Nb, cb = int(base[b]), int(L[b]), int(sizes[b]), int(caps[b])
        for dst, sc, st in ((pk, kc[b], kt[b]), (pv, vc[b], vt[b])):
            dst[:, s0:s0 + cb, :] = free
            comm = _store(normals(sc, cfg.n_kv * Lb * d), dt).reshape(cfg.n_kv, Lb, d)
            tree = _store(normals(st, cfg.n_kv * Nb * d), dt).reshape(cfg.n_kv, Nb, d)
            dst[:, s0:s0 + Lb, :] = comm.view(dst.dtype)
            dst[:, s0 + Lb:s0 + Lb + Nb, :] = tree.view(dst.dtype)
    if dt == "fp32":
        pk, pv = pk.view(np.float32), pv.view(np.float32)

    logits = _store(normals(ss["base_logits"], sumN * cfg.vocab), dt).reshape(sumN, cfg.vocab)

    pr = rng["plant"]
    if cfg.p_accept is None:
        p = pr.uniform(cfg.p_range[0], cfg.p_range[1], size=B)
    else:
        p = np.full(B, cfg.p_accept)
    plans, paths = plant_walks(T, p, pr)

    return Workload(cfg=cfg, seed=seed, lens=L, trees=T, node_off=node_off, parent=parent,
                    depth=depth, rank=rank, hidden=hidden, head_w=head_w, root_tok=root_tok,
                    q=q, pool_k=pk, pool_v=pv, seq_base=base, seq_cap=caps,
                    base_logits=logits, p_accept=p, plan=plans, plan_path=paths,
                    store_dtype=dt)


def redraw_hidden(cfg: Config, seed: int, b: int, attempt: int) -> np.ndarray:
    """A replacement last hidden state for sequence ``b``: the ``attempt``-th
    re-draw (attempt >= 1), N(0, 1) from ``SeedSequence([seed, 2, b, attempt])``,
    stored like the original row.  A test that needs a batch whose head logits
    hold no near-ties picks the attempt; the draw itself depends on nothing
    else."""
    assert attempt >= 1
    ss = np.random.SeedSequence([seed, 2, b, attempt])
    return _store(normals(ss, cfg.hidden), cfg.dtype)


def planted_logits(wl: Workload, node_tok: np.ndarray) -> np.ndarray:
    """Copy of the base logits with the planted walk written in.

    ``node_tok`` holds each tree node's token (the tree assembled from the
    heads' top-k); the planted entries sit at those tokens' columns.
    """
    return plant_logits(wl.base_logits, wl.node_off, wl.plan, node_tok, wl.store_dtype)


def plant_value(v: float, dtype: str):
    return np.float32(v) if dtype == "fp32" else to_bf16_bits(np.float32([v]))[0]


def plant_logits(base_logits: np.ndarray, node_off: np.ndarray, plans, node_tok: np.ndarray,
                 dtype: str) -> np.ndarray:
    out = base_logits.copy()
    hi, lo = plant_value(PLANT_HI, dtype), plant_value(PLANT_LO, dtype)
    for b, plan in enumerate(plans):
        o = int(node_off[b])
        for u, c, v in plan:
            out[o + u, int(node_tok[o + c])] = hi if v > 0 else lo
    return out


def storage_to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored values (fp32 or bf16 bits) to float64."""
    if dtype == "fp32":
        return x.astype(np.float64)
    return bf16_bits_to_f32(x).astype(np.float64)


# ----------------------------------------------------------------------------
# Padded batching: cache layouts with pad tokens
# ----------------------------------------------------------------------------

def padded_history(rng: np.random.Generator, real_lens: Sequence[int], steps: int, p_accept: float,
                   depth: int) -> Tuple[np.ndarray, List[np.ndarray]]:
    """The committed rows of a batch after `steps` steps of padded batching.

    Each step, sequence b commits tau_b = 1 + (levels accepted in a row, each
    with probability p_accept, at most `depth`) tokens and every sequence's
    cache grows by T = max_b tau_b rows, the last T - tau_b of them pad
    tokens.  Before those steps each cache holds its prompt (no pads), sized so
    that sequence b ends with real_lens[b] tokens.  Returns the committed rows
    per sequence and, per sequence, its flags (1 = token, 0 = pad).
    """
    B = len(real_lens)
    # tokens per step: 1 + the run of accepted levels
    runs = np.ones((steps, B), dtype=np.int64)
    alive = np.ones((steps, B), dtype=bool)
    for _ in range(depth):
        alive &= rng.random((steps, B)) < p_accept
        runs += alive
    T = runs.max(axis=1)
    gen = runs.sum(axis=0)
    prompt = np.asarray(real_lens, dtype=np.int64) - gen
    assert np.all(prompt >= 0), "fewer steps: a sequence generated more tokens than it holds"
    flags = []
    for b in range(B):
        f = [np.ones(int(prompt[b]), np.uint8)]
        for s in range(steps):
            f.append(np.concatenate([np.ones(int(runs[s, b]), np.uint8), np.zeros(int(T[s] - runs[s, b]), np.uint8)]))
        flags.append(np.concatenate(f))
    return np.array([len(f) for f in flags], dtype=np.int32), flags


def pool_key_flags(wl: Workload, slab_flags: Sequence[np.ndarray]) -> np.ndarray:
    """Per pool row flags from per-slab flags of the committed rows; every other
    row (tree rows, free rows, canaries) is flagged 0: those are never read as
    committed keys."""
    f = np.zeros(wl.cap_total, np.uint8)
    for b, sf in enumerate(slab_flags):
        assert len(sf) == int(wl.lens[b])
        s0 = int(wl.seq_base[b])
        f[s0:s0 + len(sf)] = sf
    return f



# ----------------------------------------------------------------------------
# Multi-step decoding: a pool that lives across steps, per-step model outputs
# ----------------------------------------------------------------------------

STEP_STREAMS = ("hidden", "q", "k_tree", "v_tree", "base_logits", "plant")


@dataclass
class DecodeSetup:
    cfg: Config
    seed: int
    lens: np.ndarray            # int32 [B] committed rows before the first step
    seq_base: np.ndarray        # int64 [B]
    seq_cap: np.ndarray         # int32 [B] slab rows: the budget of the whole run
    pool_k: np.ndarray          # [n_kv, cap_total, d] stored, committed rows filled
    pool_v: np.ndarray
    default: Tree               # default tree, pruned each step to the slab's free rows
    head_w: np.ndarray          # [n_heads, vocab, hidden]
    w1: np.ndarray | None       # [n_heads, hidden, hidden] residual blocks, or None
    b1: np.ndarray | None       # [n_heads, hidden]
    root_tok: np.ndarray        # int32 [B] first step's root tokens
    p_accept: np.ndarray        # float64 [B] planted acceptance per level
    temperature: float | None   # sampled next token at this temperature, or greedy (None)
    sample_seed: int
    typical: tuple | None = None  # (temperature, eps, delta): typical acceptance; None: greedy

    @property
    def cap_total(self) -> int:
        return int(self.pool_k.shape[1])


@dataclass
class StepInputs:
    hidden: np.ndarray          # [len(seqs), hidden] the base model's last hidden states
    q: np.ndarray               # [sumN, n_q, d]
    tree_k: np.ndarray          # [n_kv, sumN, d] K/V rows of the tree nodes, node order
    tree_v: np.ndarray
    base_logits: np.ndarray     # [sumN, vocab] before planting
    plans: list                 # planted walks per active sequence


def decode_setup(cfg: Config, seed: int, default: Tree, room: Sequence[int], resblock: bool = True,
                 temperature: float | None = 0.8, lens: Sequence[int] | None = None,
                 head_w: np.ndarray | None = None, typical: tuple | None = None) -> DecodeSetup:
    """Initial state of a multi-step run: each slab holds its committed rows
    and room[b] free rows for the whole run (head_w: reuse these head weights;
    typical: (temperature, eps, delta) of typical acceptance, else greedy)."""
    ss = dict(zip(STREAMS, np.random.SeedSequence(seed).spawn(len(STREAMS))))
    rng = {k: np.random.Generator(np.random.PCG64(v)) for k, v in ss.items()}
    B, d, dt = cfg.B, cfg.head_dim, cfg.dtype
    L = _lens(cfg, rng["lens"]) if lens is None else np.asarray(lens, np.int32)
    caps = (L.astype(np.int64) + np.asarray(room, np.int64)).astype(np.int32)
    base = np.zeros(B, dtype=np.int64)
    row = 1
    for b in range(B):
        base[b] = row
        row += int(caps[b]) + 1
    if dt == "fp32":
        pk = np.full((cfg.n_kv, row, d), CANARY_FP32, dtype=np.uint32)
        free = FREE_FP32
    else:
        pk = np.full((cfg.n_kv, row, d), CANARY_BF16, dtype=np.uint16)
        free = FREE_BF16
    pv = pk.copy()
    kc, vc = ss["k_comm"].spawn(B), ss["v_comm"].spawn(B)
    for b in range(B):
        s0, Lb, cb = int(base[b]), int(L[b]), int(caps[b])
        for dst, sc in ((pk, kc[b]), (pv, vc[b])):
            dst[:, s0:s0 + cb, :] = free
            dst[:, s0:s0 + Lb, :] = _store(normals(sc, cfg.n_kv * Lb * d), dt).reshape(cfg.n_kv, Lb, d).view(dst.dtype)
    if dt == "fp32":
        pk, pv = pk.view(np.float32), pv.view(np.float32)
    hw = ss["head_w"].spawn(3)
    if head_w is None:
        head_w = _store(normals(hw[0], cfg.n_heads * cfg.vocab * cfg.hidden, cfg.w_std), dt)
        head_w = head_w.reshape(cfg.n_heads, cfg.vocab, cfg.hidden)
    w1 = b1 = None
    if resblock:
        w1 = _store(normals(hw[1], cfg.n_heads * cfg.hidden * cfg.hidden, cfg.w_std), dt)
        w1 = w1.reshape(cfg.n_heads, cfg.hidden, cfg.hidden)
        b1 = _store(normals(hw[2], cfg.n_heads * cfg.hidden, cfg.w_std), dt).reshape(cfg.n_heads, cfg.hidden)
    root = rng["root"].integers(0, cfg.vocab, size=B).astype(np.int32)
    pr = rng["plant"]
    p = pr.uniform(cfg.p_range[0], cfg.p_range[1], size=B) if cfg.p_accept is None else np.full(B, cfg.p_accept)
    return DecodeSetup(cfg=cfg, seed=seed, lens=L, seq_base=base, seq_cap=caps, pool_k=pk, pool_v=pv,
                       default=default, head_w=head_w, w1=w1, b1=b1, root_tok=root, p_accept=p,
                       temperature=temperature, sample_seed=seed * 7919 + 17, typical=typical)


def tree_prefix(t: Tree, n: int) -> Tree:
    """The first n nodes of a breadth-first tree (a tree again)."""
    return Tree(t.parent[:n].copy(), t.depth[:n].copy(), t.rank[:n].copy())


def decode_step_inputs(setup: DecodeSetup, step: int, seqs: Sequence[int], trees: Sequence[Tree]) -> StepInputs:
    """The base model's outputs for one step of the active sequences `seqs`
    (Gaussian stand-ins, drawn from (seed, step)), and the planted walks."""
    cfg, dt, d = setup.cfg, setup.cfg.dtype, setup.cfg.head_dim
    ss = dict(zip(STEP_STREAMS, np.random.SeedSequence([setup.seed, 1 + step]).spawn(len(STEP_STREAMS))))
    n = [t.n for t in trees]
    sumN = int(sum(n))
    hidden = _store(normals(ss["hidden"], len(seqs) * cfg.hidden), dt).reshape(len(seqs), cfg.hidden)
    q = _store(normals(ss["q"], sumN * cfg.n_q * d), dt).reshape(sumN, cfg.n_q, d)
    tk = _store(normals(ss["k_tree"], cfg.n_kv * sumN * d), dt).reshape(cfg.n_kv, sumN, d)
    tv = _store(normals(ss["v_tree"], cfg.n_kv * sumN * d), dt).reshape(cfg.n_kv, sumN, d)
    lg = _store(normals(ss["base_logits"], sumN * cfg.vocab), dt).reshape(sumN, cfg.vocab)
    plans, _ = plant_walks(list(trees), setup.p_accept[list(seqs)],
                           np.random.Generator(np.random.PCG64(ss["plant"])))
    return StepInputs(hidden=hidden, q=q, tree_k=tk, tree_v=tv, base_logits=lg, plans=plans)
