"""One verify step on the GPU through the C ABI.

``VerifyStep`` uploads a synthetic workload (torch tensors for device memory),
allocates outputs and workspaces once, and runs the four stages in order on the
current torch stream.  All arithmetic runs in libspecmemo's kernels.
"""

from __future__ import annotations

import numpy as np
import torch

from . import specmemo as sm
from .synth import Workload


def to_device(x: np.ndarray, dtype: str, device) -> torch.Tensor:
    """Stored array (float32, or uint16 bf16 bits) -> device tensor of that type
    (a tensor already on the device passes through)."""
    if isinstance(x, torch.Tensor):
        return x
    if dtype == "fp32":
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device)
    t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(device)
    return t.view(torch.bfloat16)


def to_host_storage(t: torch.Tensor, dtype: str) -> np.ndarray:
    """Device tensor -> stored array (float32, or uint16 bf16 bits)."""
    t = t.detach().cpu()
    if dtype == "fp32":
        return t.numpy()
    return t.view(torch.int16).numpy().view(np.uint16)


class VerifyStep:
    def __init__(self, wl: Workload, device="cuda", mode: int = sm.GREEDY, temperature: float = 0.7,
                 eps: float = 0.09, delta: float = 0.3, keep_logits: bool = False, pack_heads: bool = True,
                 key_valid: np.ndarray | None = None):
        """key_valid: per pool row flags (0 = pad token) for the padded-batching
        variant (tree_attn_padded / kv_pad_update); None for the ragged path."""
        cfg = wl.cfg
        self.wl, self.cfg, self.device = wl, cfg, device
        self.dt = sm.FP32 if cfg.dtype == "fp32" else sm.BF16
        self.mode, self.temperature, self.eps, self.delta = mode, temperature, eps, delta
        i32 = dict(dtype=torch.int32, device=device)
        self.trees = sm.Trees(wl.node_off, wl.parent, wl.depth, wl.rank, device=device)
        self.h = to_device(wl.hidden, cfg.dtype, device)
        self.head_w = to_device(wl.head_w, cfg.dtype, device) if wl.head_w is not None else None
        # bf16 heads are packed once into the projection's streaming order (a
        # load-time step: the heads are fixed for a model)
        self.head_layout = sm.HEADS_ROWMAJOR
        if pack_heads and self.head_w is not None and self.dt == sm.BF16:
            nb = sm.packed_heads_bytes(self.dt, cfg.n_heads, cfg.vocab, cfg.hidden)
            packed = torch.empty(nb, dtype=torch.uint8, device=device)
            sm.pack_heads(self.dt, cfg.n_heads, cfg.vocab, cfg.hidden, self.head_w, packed)
            self.head_w, self.head_layout = packed, sm.HEADS_PACKED
        self.root_tok = torch.from_numpy(wl.root_tok.copy()).to(device)
        self.q = to_device(wl.q, cfg.dtype, device)
        self.k = to_device(wl.pool_k, cfg.dtype, device)
        self.v = to_device(wl.pool_v, cfg.dtype, device)
        self.seq_len = torch.from_numpy(wl.lens.copy()).to(device)
        self.kv = sm.KVPool(self.k, self.v, self.seq_len, wl.seq_base, wl.seq_cap, wl.lens)
        B, nh, kmax, total = cfg.B, cfg.n_heads, cfg.kmax, wl.total_nodes
        self.logits = torch.empty((B, nh, cfg.vocab), dtype=torch.float32, device=device) if keep_logits else None
        self.topk_ids = torch.empty((B, nh, kmax), **i32)
        self.topk_vals = torch.empty((B, nh, kmax), dtype=torch.float32, device=device)
        self.node_tok = torch.empty(total, **i32)
        self.out = torch.empty_like(self.q)
        self.path_stride = cfg.n_heads + 1
        self.accept_len = torch.empty(B, **i32)
        self.path = torch.empty((B, self.path_stride), **i32)
        self.next_tok = torch.empty(B, **i32)
        self.base_logits = None
        self.key_valid = self.pos = None
        if key_valid is not None:
            words = sm.pack_key_valid(key_valid)
            self.key_valid = torch.from_numpy(words.view(np.int32)).to(device)
            # position of each sequence's next token: its committed rows minus the pads
            kv_flags = np.asarray(key_valid) != 0
            pos = [int(kv_flags[int(wl.seq_base[b]):int(wl.seq_base[b]) + int(wl.lens[b])].sum()) for b in range(B)]
            self.pos = torch.tensor(pos, dtype=torch.int32, device=device)
        ws = max(sm.workspace_bytes(sm.WS_TOPK, self.dt, self.trees, None, nh, cfg.vocab),
                 sm.workspace_bytes(sm.WS_ACCEPT, self.dt, self.trees, None, sm.TYPICAL),
                 sm.workspace_bytes(sm.WS_PAD, self.dt, self.trees, None, 0) if key_valid is not None else 0)
        self.ws_bytes = ws
        self.ws = torch.empty(max(ws, 16), dtype=torch.uint8, device=device)
        # the attention has a workspace of its own: it may run concurrently with the projection
        self.ws_attn_bytes = max(sm.workspace_bytes(sm.WS_ATTN, self.dt, self.trees, self.kv, cfg.n_q), 16)
        self.ws_attn = torch.empty(self.ws_attn_bytes, dtype=torch.uint8, device=device)
        self.side_box = [None]    # the second stream of run_overlapped, shared with replicas

    def replica(self) -> "VerifyStep":
        """Another step over the same workload that shares the head weights,
        trees and hidden states but owns copies of every per-step buffer
        (queries, pool, lengths, base logits, outputs, workspace).  Steps
        rotated over enough replicas find none of their data in the caches."""
        import copy
        r = copy.copy(self)
        for name in ("q", "k", "v", "seq_len", "out", "topk_ids", "topk_vals", "node_tok", "accept_len", "path",
                     "next_tok", "ws", "ws_attn", "base_logits", "logits", "key_valid", "pos"):
            t = getattr(self, name)
            if t is not None:
                setattr(r, name, t.clone())
        r.kv = sm.KVPool(r.k, r.v, r.seq_len, self.wl.seq_base, self.wl.seq_cap, self.wl.lens)
        return r

    def step_bytes(self) -> int:
        """Device bytes a replica owns (what one step touches besides the heads)."""
        ts = (self.q, self.k, self.v, self.out, self.base_logits, self.ws, self.ws_attn, self.topk_ids, self.node_tok)
        return int(sum(t.numel() * t.element_size() for t in ts if t is not None))

    def set_base_logits(self, stored: np.ndarray):
        self.base_logits = to_device(stored, self.cfg.dtype, self.device)

    # ---- stages -------------------------------------------------------------------
    def medusa_topk(self, stream=None):
        c = self.cfg
        sm.medusa_topk(self.dt, self.trees, c.hidden, c.vocab, c.n_heads, c.topk, self.h, self.head_w,
                       self.root_tok, self.topk_ids, self.node_tok, logits_out=self.logits,
                       topk_vals=self.topk_vals, ws=self.ws, ws_bytes=self.ws_bytes, stream=stream,
                       head_layout=self.head_layout)

    def tree_attn(self, stream=None):
        sm.tree_attn(self.dt, self.trees, self.kv, self.cfg.n_q, self.q, self.out, ws=self.ws_attn,
                     ws_bytes=self.ws_attn_bytes, stream=stream)

    def accept(self, stream=None):
        sm.accept(self.dt, self.trees, self.cfg.vocab, self.mode, self.base_logits, self.node_tok,
                  self.accept_len, self.path, self.path_stride, self.next_tok, temperature=self.temperature,
                  eps=self.eps, delta=self.delta, ws=self.ws, ws_bytes=self.ws_bytes, stream=stream)

    def kv_compact(self, stream=None):
        sm.kv_compact(self.dt, self.trees, self.kv, self.accept_len, self.path, self.path_stride, stream=stream)

    def accept_compact(self, stream=None):
        """Acceptance and compaction in one call (the fused entry point)."""
        sm.accept_compact(self.dt, self.trees, self.kv, self.cfg.vocab, self.mode, self.base_logits, self.node_tok,
                          self.accept_len, self.path, self.path_stride, self.next_tok, temperature=self.temperature,
                          eps=self.eps, delta=self.delta, ws=self.ws, ws_bytes=self.ws_bytes, stream=stream)

    def reset_pool(self):
        """Restore the workload's pool and committed lengths on the device."""
        c = self.cfg
        self.k.copy_(to_device(self.wl.pool_k, c.dtype, self.device))
        self.v.copy_(to_device(self.wl.pool_v, c.dtype, self.device))
        self.seq_len.copy_(torch.from_numpy(self.wl.lens.copy()))

    def tree_attn_padded(self, stream=None):
        sm.tree_attn_padded(self.dt, self.trees, self.kv, self.key_valid, self.cfg.n_q, self.q, self.out,
                            ws=self.ws_attn, ws_bytes=self.ws_attn_bytes, stream=stream)

    def kv_pad_update(self, stream=None):
        sm.kv_pad_update(self.dt, self.trees, self.kv, self.accept_len, self.path, self.path_stride, self.key_valid,
                         self.pos, ws=self.ws, ws_bytes=self.ws_bytes, stream=stream)

    def run(self, stream=None):
        self.medusa_topk(stream)
        self.tree_attn(stream)
        self.accept(stream)
        self.kv_compact(stream)

    def run_fused(self, stream=None):
        """The step with acceptance and compaction fused into one call."""
        self.medusa_topk(stream)
        self.tree_attn(stream)
        self.accept_compact(stream)

    def run_overlapped(self):
        """The fused step with the attention on a second stream, concurrent
        with the head projection and top-k.  The two stages share no data: the
        attention reads queries and K/V, the projection hidden states and head
        weights.  The side stream first waits for the main stream (the
        previous step's compaction rewrites K/V rows the attention reads), and
        the main stream waits for the attention before the acceptance and
        compaction.  Both streams have the default priority."""
        main = torch.cuda.current_stream(self.device)
        if self.side_box[0] is None:
            self.side_box[0] = torch.cuda.Stream(device=self.device)
        side = self.side_box[0]
        side.wait_stream(main)
        with torch.cuda.stream(side):
            self.tree_attn()
        self.medusa_topk()
        main.wait_stream(side)
        self.accept_compact()

    def run_padded(self, stream=None):
        """The step of the padded-batching variant: pad tokens masked in
        attention, accepted tokens padded to the batch's longest acceptance."""
        self.medusa_topk(stream)
        self.tree_attn_padded(stream)
        self.accept(stream)
        self.kv_pad_update(stream)


class DecodeLoop:
    """Multi-step decoding through the library on one GPU.

    The KV pool lives on the device across steps.  Per step: tree sizes from
    the library's planner (the default tree pruned to each slab's free rows; a
    full slab ends its sequence), the step's model outputs uploaded (the tree's
    K/V rows written at slab rows L_b ..), residual-block heads and the
    projection with top-k, the planted base-model logits (written on the device
    at the tokens the heads chose), tree attention, greedy or typical
    acceptance with the compaction (one call), the next token (the
    acceptance's or sampled).  The host reads back the
    accepted lengths and next tokens once per step: they size the next step.
    """

    def __init__(self, setup, device="cuda", keep_logits: bool = True, timing: bool = False):
        cfg = setup.cfg
        self.timing, self.events = timing, []
        self.setup, self.cfg, self.device, self.keep_logits = setup, cfg, device, keep_logits
        self.dt = sm.FP32 if cfg.dtype == "fp32" else sm.BF16
        self.k = to_device(setup.pool_k, cfg.dtype, device)
        self.v = to_device(setup.pool_v, cfg.dtype, device)
        head_w = to_device(setup.head_w, cfg.dtype, device)
        self.head_layout = sm.HEADS_ROWMAJOR
        if self.dt == sm.BF16:
            packed = torch.empty(sm.packed_heads_bytes(self.dt, cfg.n_heads, cfg.vocab, cfg.hidden),
                                 dtype=torch.uint8, device=device)
            sm.pack_heads(self.dt, cfg.n_heads, cfg.vocab, cfg.hidden, head_w, packed)
            head_w, self.head_layout = packed, sm.HEADS_PACKED
        self.head_w = head_w
        self.w1 = self.b1 = None
        if setup.w1 is not None:
            w1 = to_device(setup.w1, cfg.dtype, device)
            self.w1_layout = sm.HEADS_ROWMAJOR
            if self.dt == sm.BF16:
                packed = torch.empty(sm.packed_heads_bytes(self.dt, cfg.n_heads, cfg.hidden, cfg.hidden),
                                     dtype=torch.uint8, device=device)
                sm.pack_heads(self.dt, cfg.n_heads, cfg.hidden, cfg.hidden, w1, packed)
                w1, self.w1_layout = packed, sm.HEADS_PACKED
            self.w1 = w1
            self.b1 = to_device(setup.b1, cfg.dtype, device)
        self.lens = setup.lens.astype(np.int32).copy()
        self.root = setup.root_tok.astype(np.int32).copy()
        self.stride = cfg.n_heads + 1
        d = setup.default
        self.default = (np.asarray(d.parent, np.int32), np.asarray(d.depth, np.int32), np.asarray(d.rank, np.int32))
        from .synth import PLANT_HI, PLANT_LO
        self._plant_hi, self._plant_lo = PLANT_HI, PLANT_LO   # the input generator's planted logits
        self._tree_cache = {}
        self.mode = sm.GREEDY if setup.typical is None else sm.TYPICAL
        self.typical = {} if setup.typical is None else dict(zip(("temperature", "eps", "delta"), setup.typical))
        self._pin = [(None, None), (None, None)]

    def plan(self):
        """Active sequences and their tree sizes for the next step."""
        sizes = sm.plan_tree_sizes(self.lens, self.setup.seq_cap, len(self.default[0]))
        seqs = [b for b in range(self.cfg.B) if sizes[b] > 0]
        return seqs, [int(sizes[b]) for b in seqs]

    def _tree_arrays(self, sizes):
        """The step's trees (prefixes of the default tree) as a library tree
        batch with its device arrays, and the size of the projection's and
        acceptance's workspace; kept per size tuple (most steps repeat one)."""
        key = tuple(sizes)
        hit = self._tree_cache.get(key)
        if hit is None:
            from . import synth
            trees = [synth.tree_prefix(synth.Tree(*self.default), n) for n in sizes]
            node_off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
            host = [node_off] + [np.concatenate([getattr(tr, f) for tr in trees]).astype(np.int32)
                                 for f in ("parent", "depth", "rank")]
            dev = torch.from_numpy(np.concatenate(host)).pin_memory().to(self.device, non_blocking=True)
            tr = sm.Trees(*host, dev_arrays=list(dev.split([len(a) for a in host])))
            ws = max(sm.workspace_bytes(sm.WS_TOPK, self.dt, tr, None, self.cfg.n_heads, self.cfg.vocab),
                     sm.workspace_bytes(sm.WS_ACCEPT, self.dt, tr, None, self.mode))
            hit = (trees, tr, ws)
            if len(self._tree_cache) < 256:
                self._tree_cache[key] = hit
        return hit

    def _upload(self, slot: int, parts):
        """Concatenate int32 arrays into pinned host memory and copy them to
        the device asynchronously (two independent slots); returns the device
        buffer.  A slot's host memory is rewritten only after the previous
        step's read-back, which waits for its copy."""
        n = sum(len(a) for a in parts)
        pin, dbuf = self._pin[slot]
        if pin is None or pin.numel() < n:
            cap = max(n, 2 * (0 if pin is None else pin.numel()))
            pin = torch.empty(cap, dtype=torch.int32, pin_memory=True)
            dbuf = torch.empty(cap, dtype=torch.int32, device=self.device)
            self._pin[slot] = (pin, dbuf)
        np.concatenate(parts, out=pin.numpy()[:n])
        dbuf[:n].copy_(pin[:n], non_blocking=True)
        return dbuf

    def phase_ms(self):
        """Per-step stage times (ms) from the events of the steps run with
        timing on."""
        out = []
        for ev in self.events:
            names = list(ev)
            out.append({b: ev[a].elapsed_time(ev[b]) for a, b in zip(names, names[1:])})
        return out

    def step(self, t: int, inputs=None, record: bool = True, plan=None):
        """One step; returns its record (host copies when `record`), or None when
        every slab is full.  The launches come in the order that keeps the
        device busy: the residual blocks (they need only the hidden states),
        the projection and top-k (after a small upload of the roots and
        lengths), then the model outputs' writes, attention, acceptance with
        compaction (one call) and the sampled next token.  The accepted
        lengths and next tokens come back in one read-back.  `plan`, when
        given, is what plan() returns for the current lengths."""
        from . import synth
        cfg, st, dev = self.cfg, self.setup, self.device
        seqs, sizes = self.plan() if plan is None else plan
        if not seqs:
            return None
        if inputs is None:
            inputs = synth.decode_step_inputs(st, t, seqs, self._tree_arrays(sizes)[0])
        inp = inputs
        B = len(seqs)
        s = torch.cuda.current_stream().cuda_stream
        i32 = dict(dtype=torch.int32, device=dev)
        ev = {}

        def mark(name):
            if self.timing:
                e = torch.cuda.Event(enable_timing=True)
                e.record()
                ev[name] = e

        h = to_device(inp.hidden, cfg.dtype, dev)
        mark("start")
        layout = self.head_layout
        if self.w1 is not None:
            hh = torch.empty((cfg.n_heads, B, cfg.hidden), dtype=h.dtype, device=dev)
            sm.medusa_resblock(self.dt, B, cfg.hidden, cfg.n_heads, h, self.w1, self.b1, hh,
                               w1_layout=self.w1_layout, stream=s)
            h, layout = hh, layout | sm.HEADS_INPUT_PER_HEAD
        mark("resblock")
        trees, tr, ws_fixed = self._tree_arrays(sizes)
        node_off = tr.node_off_h
        sumN = int(node_off[-1])
        base, L, caps = st.seq_base[seqs], self.lens[seqs].copy(), st.seq_cap[seqs]
        small = self._upload(0, [self.root[seqs].astype(np.int32), L.astype(np.int32)])
        root, seq_len = small[:B], small[B:2 * B]
        kv = sm.KVPool(self.k, self.v, seq_len, base, caps, L)
        mark("upload")
        logits = torch.empty((B, cfg.n_heads, cfg.vocab), dtype=torch.float32, device=dev) if self.keep_logits else None
        ws_bytes = max(ws_fixed, sm.workspace_bytes(sm.WS_ATTN, self.dt, tr, kv, cfg.n_q),
                       sm.workspace_bytes(sm.WS_SAMPLE, self.dt, tr, None, 0, cfg.vocab), 16)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        ids = torch.empty((B, cfg.n_heads, cfg.kmax), **i32)
        tok = torch.empty(sumN, **i32)
        sm.medusa_topk(self.dt, tr, cfg.hidden, cfg.vocab, cfg.n_heads, cfg.topk, h, self.head_w, root, ids, tok,
                       logits_out=logits, ws=ws, ws_bytes=ws_bytes, head_layout=layout, stream=s)
        mark("medusa_topk")
        # The base model's outputs, written while the projection runs: the
        # tree's K/V rows at slab rows seq_base + L + local index, the logits
        # with the planted walk at the tokens the heads chose.
        rows = (np.repeat(base.astype(np.int64) + L - node_off[:-1], sizes) + np.arange(sumN)).astype(np.int32)
        cnt = [len(p) for p in inp.plans]
        plant = np.array([(u, c, 1 if val > 0 else 0) for p in inp.plans for (u, c, val) in p],
                         np.int32).reshape(-1, 3)
        if plant.size:
            shift = np.repeat(node_off[:-1], cnt)
            plant[:, 0] += shift
            plant[:, 1] += shift
        big = self._upload(1, [rows, np.ascontiguousarray(plant.T).reshape(-1)])
        ri = big[:sumN].to(torch.int64)
        self.k.index_copy_(1, ri, to_device(inp.tree_k, cfg.dtype, dev))
        self.v.index_copy_(1, ri, to_device(inp.tree_v, cfg.dtype, dev))
        lg = to_device(inp.base_logits, cfg.dtype, dev)
        if plant.size:
            plant_d = big[sumN:sumN + plant.size].view(3, -1)
            cols = tok[plant_d[1].to(torch.int64)].to(torch.int64)
            vals = torch.where(plant_d[2] > 0, float(self._plant_hi), float(self._plant_lo)).to(lg.dtype)
            lg[plant_d[0].to(torch.int64), cols] = vals
        # attention, acceptance, next token, compaction
        q = to_device(inp.q, cfg.dtype, dev)
        out = torch.empty_like(q)
        mark("model")
        sm.tree_attn(self.dt, tr, kv, cfg.n_q, q, out, ws=ws, ws_bytes=ws_bytes, stream=s)
        mark("tree_attn")
        res = torch.empty((2, B), **i32)            # accepted lengths, next tokens: read back together
        acc, nxt = res[0], res[1]
        path = torch.empty((B, self.stride), **i32)
        # acceptance with the compaction fused in; the sampled next token reads
        # only the logits and the accepted path, so it may follow the compaction
        sm.accept_compact(self.dt, tr, kv, cfg.vocab, self.mode, lg, tok, acc, path, self.stride, nxt, ws=ws,
                          ws_bytes=ws_bytes, stream=s, **self.typical)
        mark("accept_compact")
        if st.temperature is not None:
            sm.sample_next(self.dt, tr, cfg.vocab, st.temperature, st.sample_seed, t, lg, acc, path, self.stride, nxt,
                           ws=ws, ws_bytes=ws_bytes, stream=s)
        mark("sample_next")
        res_h = res.cpu().numpy()
        acc_h, nxt_h = res_h[0].copy(), res_h[1].copy()
        if self.timing:
            self.events.append(ev)
        self.lens[seqs] = L + acc_h + 1
        self.root[seqs] = nxt_h
        rec = dict(step=t, seqs=seqs, sizes=sizes, acc=acc_h, next_tok=nxt_h, lens=self.lens.copy())
        if record:
            rec.update(z=None if logits is None else logits.cpu().numpy(), ids=ids.cpu().numpy(),
                       tok=tok.cpu().numpy(), attn=out, path=path.cpu().numpy(), seq_len=seq_len.cpu().numpy())
        return rec
