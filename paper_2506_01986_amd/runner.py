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
    """Stored array (float32, or uint16 bf16 bits) -> device tensor of that type."""
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
                 sm.workspace_bytes(sm.WS_ATTN, self.dt, self.trees, self.kv, cfg.n_q),
                 sm.workspace_bytes(sm.WS_ACCEPT, self.dt, self.trees, None, mode),
                 sm.workspace_bytes(sm.WS_PAD, self.dt, self.trees, None, 0) if key_valid is not None else 0)
        self.ws_bytes = ws
        self.ws = torch.empty(max(ws, 16), dtype=torch.uint8, device=device)

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
        sm.tree_attn(self.dt, self.trees, self.kv, self.cfg.n_q, self.q, self.out, ws=self.ws,
                     ws_bytes=self.ws_bytes, stream=stream)

    def accept(self, stream=None):
        sm.accept(self.dt, self.trees, self.cfg.vocab, self.mode, self.base_logits, self.node_tok,
                  self.accept_len, self.path, self.path_stride, self.next_tok, temperature=self.temperature,
                  eps=self.eps, delta=self.delta, ws=self.ws, ws_bytes=self.ws_bytes, stream=stream)

    def kv_compact(self, stream=None):
        sm.kv_compact(self.dt, self.trees, self.kv, self.accept_len, self.path, self.path_stride, stream=stream)

    def tree_attn_padded(self, stream=None):
        sm.tree_attn_padded(self.dt, self.trees, self.kv, self.key_valid, self.cfg.n_q, self.q, self.out, ws=self.ws,
                            ws_bytes=self.ws_bytes, stream=stream)

    def kv_pad_update(self, stream=None):
        sm.kv_pad_update(self.dt, self.trees, self.kv, self.accept_len, self.path, self.path_stride, self.key_valid,
                         self.pos, ws=self.ws, ws_bytes=self.ws_bytes, stream=stream)

    def run(self, stream=None):
        self.medusa_topk(stream)
        self.tree_attn(stream)
        self.accept(stream)
        self.kv_compact(stream)

    def run_padded(self, stream=None):
        """The step of the padded-batching variant: pad tokens masked in
        attention, accepted tokens padded to the batch's longest acceptance."""
        self.medusa_topk(stream)
        self.tree_attn_padded(stream)
        self.accept(stream)
        self.kv_pad_update(stream)
